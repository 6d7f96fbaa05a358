"""End-to-end use of the optimizer: a GPT with the 160M model's block shapes
(d_model 768, 4 of its 12 blocks here to keep the test short) trained on
synthetic tokens with CurvaDion on every block matrix and AdamW on the
embedding and norms (the paper's setup hands Dion the weight matrices).

The token stream is learnable (each token is its predecessor plus one, from a
random start), so the loss must fall well below its start, ln(512).  The test also
prints the optimizer step time of CurvaDion next to torch's fused AdamW over
the same matrices.  Everything runs in fp32."""
import math
import time

import pytest
import torch
import torch.nn.functional as F

from paper_2512_13728_amd.optim import CurvaDion

pytestmark = pytest.mark.gpu
DEV = "cuda"
D, HEADS, BLOCKS, VOCAB, SEQ, BATCH = 768, 12, 4, 512, 128, 16


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield


class Block(torch.nn.Module):
    def __init__(self):
        super().__init__()
        self.n1, self.n2 = torch.nn.RMSNorm(D), torch.nn.RMSNorm(D)
        self.qkv = torch.nn.Linear(D, 3 * D, bias=False)   # weight 2304 x 768
        self.o = torch.nn.Linear(D, D, bias=False)
        self.fc = torch.nn.Linear(D, 4 * D, bias=False)
        self.proj = torch.nn.Linear(4 * D, D, bias=False)

    def forward(self, x, mask):
        b, t, _ = x.shape
        q, k, v = self.qkv(self.n1(x)).view(b, t, 3, HEADS, D // HEADS).permute(2, 0, 3, 1, 4)
        att = (q @ k.transpose(-1, -2).contiguous()) / math.sqrt(D // HEADS)
        att = att.masked_fill(mask, float("-inf")).softmax(-1)
        x = x + self.o((att @ v).transpose(1, 2).reshape(b, t, D))
        return x + self.proj(F.relu(self.fc(self.n2(x))).square())


class GPT(torch.nn.Module):
    def __init__(self):
        super().__init__()
        self.emb = torch.nn.Embedding(VOCAB, D)
        torch.nn.init.normal_(self.emb.weight, std=0.02)
        self.blocks = torch.nn.ModuleList(Block() for _ in range(BLOCKS))
        self.norm = torch.nn.RMSNorm(D)

    def forward(self, idx):
        t = idx.shape[1]
        mask = torch.triu(torch.ones(t, t, dtype=torch.bool, device=idx.device), 1)
        x = self.emb(idx)
        for blk in self.blocks:
            x = blk(x, mask)
        return self.norm(x) @ self.emb.weight.T      # tied output head


def _batch(gen):
    """Tokens x_t = (x_0 + t) mod VOCAB from a random x_0 per sequence."""
    start = torch.randint(0, VOCAB, (BATCH, 1), generator=gen)
    idx = (start + torch.arange(SEQ + 1)[None, :]) % VOCAB
    idx = idx.to(DEV)
    return idx[:, :-1], idx[:, 1:]


def _time_step(opt, params, reps=5):
    for p in params:
        p.grad = torch.randn_like(p) * 1e-3
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        opt.step()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / reps * 1e3


def test_gpt_blocks_train_and_step_cost():
    torch.manual_seed(0)
    model = GPT().to(DEV)
    mats = [p for n, p in model.named_parameters() if n.startswith("blocks") and p.dim() == 2]
    rest = [p for n, p in model.named_parameters() if not (n.startswith("blocks") and p.dim() == 2)]
    assert len(mats) == 4 * BLOCKS
    opt = CurvaDion(mats, lr=0.02, momentum=0.95, rank=0.125, tau=0.5, weight_decay=0.01)
    aux = torch.optim.AdamW(rest, lr=3e-3, weight_decay=0.0)
    gen = torch.Generator().manual_seed(1)
    losses, syncs = [], 0
    for step in range(60):
        x, y = _batch(gen)
        logits = model(x)
        loss = F.cross_entropy(logits.reshape(-1, VOCAB), y.reshape(-1))
        opt.zero_grad(set_to_none=False)
        aux.zero_grad()
        loss.backward()
        opt.step()
        aux.step()
        losses.append(loss.item())
        syncs += int(opt.last[torch.float32][1])
    first, last = sum(losses[:5]) / 5, sum(losses[-5:]) / 5
    # optimizer step cost over the 16 block matrices (7.1M params each block)
    ms_cd = _time_step(opt, mats)
    ref = [torch.nn.Parameter(p.detach().clone()) for p in mats]
    adam = torch.optim.AdamW(ref, lr=1e-3, fused=True)
    ms_adam = _time_step(adam, ref)
    print(f"loss {first:.3f} -> {last:.3f} in 60 steps ({syncs} syncs); optimizer step over "
          f"{sum(p.numel() for p in mats) / 1e6:.1f}M matrix params: CurvaDion {ms_cd:.3f} ms, "
          f"fused AdamW {ms_adam:.3f} ms", flush=True)
    assert abs(losses[0] - math.log(VOCAB)) < 1.0
    assert math.isfinite(last) and last < 0.5 * first
    assert syncs >= 1
