// Prints the streaming-pass launch plan of the C ABI for the layer shapes read
// from stdin ("m n" per line): one line per launch, "<layers> <blocks>".
// Built by the CPU tests with a plain C++ compiler against the library's
// planning header (it has no HIP dependency).
#include <cstdio>
#include <vector>

#include "plan.hpp"

int main() {
  std::vector<long long> numel;
  long long m, n;
  while (std::scanf("%lld %lld", &m, &n) == 2) numel.push_back(m * n);
  const auto plan = cd::plan_stream_batches(numel, cd::MAXS, cd::MAX_STREAM_BLOCKS, cd::FORM_CHUNK);
  for (const auto& b : plan) {
    long long blocks = 0;
    for (int i : b) blocks += (numel[i] + cd::FORM_CHUNK - 1) / cd::FORM_CHUNK;
    std::printf("%zu %lld\n", b.size(), blocks);
  }
  return 0;
}
