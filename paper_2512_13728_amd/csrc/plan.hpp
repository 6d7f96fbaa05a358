// Host-side launch planning of the C ABI: pure functions of the layer sizes,
// with no HIP dependency, so that the CPU tests compile and check them with
// a plain C++ compiler.
#pragma once

#include <vector>

namespace cd {

constexpr int MAXB = 32;          // layers per batched launch of the sync branch (one shape)
// Streaming-pass launches (any shapes): at most MAXS layers and 98304 blocks
// of 4096 elements (402.7M elements, 7.25 GB of M, X and bf16 G with the
// fused skip update).  The 1.3B-shaped set then splits into 3 x 32 layers
// (eight transformer blocks of 12288 blocks each per launch); launches of 48
// or 64 layers (600-800M elements) streamed 1.7% slower there.  The
// 160M-shaped set (48 layers, 20736 blocks) runs as one launch, 3.4% faster
// than two.
constexpr int MAXS = 48;
constexpr long long MAX_STREAM_BLOCKS = 98304;   // x 4096 elements
constexpr int NTHREADS = 256;     // threads per block for the streaming kernels
// Every block of a streaming pass covers FORM_CHUNK consecutive elements of
// one layer.
constexpr int FORM_CHUNK = NTHREADS * 4 * 4;   // 4096 elements

// Launches of the streaming passes (buffer formation, local update): layers
// in group order, each launch taking whole layers until it holds max_layers
// layers or one more layer would take it past max_blocks blocks of `chunk`
// elements.  A layer larger than max_blocks gets a launch of its own.
inline std::vector<std::vector<int>> plan_stream_batches(const std::vector<long long>& numel, int max_layers,
                                                         long long max_blocks, long long chunk) {
  std::vector<std::vector<int>> out;
  long long blocks = 0;
  for (int i = 0; i < static_cast<int>(numel.size()); ++i) {
    const long long nb = (numel[i] + chunk - 1) / chunk;
    if (out.empty() || static_cast<int>(out.back().size()) == max_layers || blocks + nb > max_blocks) {
      out.emplace_back();
      blocks = 0;
    }
    out.back().push_back(i);
    blocks += nb;
  }
  return out;
}

}  // namespace cd
