"""The largest key length the C ABI accepts, through the GPU path: one head
whose K and V each take about 2 GiB, so that the 32-bit byte offsets of a
head reach their limit. With K = 0 every score is 0 and every key gets the
same weight, so each output row is the column mean of V (a closed form the
host computes exactly, in fp64, from the same bf16 V), and the checksum
holds (no flag). A wrapped offset would read other rows of V, or zeros, and
move the mean far beyond the tolerance."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")


def _max_lk(d):
    # (Lk + 64) * d * 4 <= 2^32 - 1
    return 0xFFFFFFFF // (4 * d) - 64


def _col_mean_f64(v):
    """Exact fp64 column sums of a [Lk, d] bf16 device tensor, in chunks."""
    acc = np.zeros(v.shape[1], dtype=np.float64)
    step = 1 << 20
    for s in range(0, v.shape[0], step):
        acc += v[s:s + step].float().cpu().numpy().astype(np.float64).sum(axis=0)
    return acc / v.shape[0]


@pytest.mark.parametrize("d", [64, 128, 256])
@pytest.mark.parametrize("split", [False, True, "twopass"])
def test_uniform_weights_at_the_largest_key_length(d, split):
    Lk, Lq = _max_lk(d), 3
    print(f"[maxsize] d={d} Lk={Lk} split={split}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(7 + d)
    q = torch.randn((1, 1, Lq, d), generator=g, device="cuda").to(torch.bfloat16)
    k = torch.zeros((1, 1, Lk, d), dtype=torch.bfloat16, device="cuda")
    v = torch.randn((1, 1, Lk, d), generator=g, device="cuda").to(torch.bfloat16)
    if split == "twopass":
        o, resid, flags = F.attn_fwd_twopass(q, k, v, causal=False, scale=d ** -0.5)
    elif split:
        o, resid, flags = F.attn_fwd_splitkv(q, k, v, causal=False, scale=d ** -0.5)
    else:
        o, resid, flags = F.attn_fwd(q, k, v, causal=False, scale=d ** -0.5)
    torch.cuda.synchronize()
    mean = _col_mean_f64(v[0, 0])
    got = o[0, 0].float().cpu().numpy().astype(np.float64)
    # bf16 rounding of O (2^-9 relative) plus fp32 accumulation over Lk keys
    tol = 2.0 ** -8 * np.abs(mean) + 1e-6
    rho = (resid[0, 0].abs().cpu().numpy() / np.abs(got).sum(axis=1)).max()
    print(f"[maxsize] d={d}: max |O - mean| {np.abs(got - mean).max():.3e}, "
          f"|mean| {np.abs(mean).mean():.3e}, |r| / sum|O| {rho:.3e}", flush=True)
    assert np.all(np.abs(got - mean[None, :]) <= tol[None, :]), np.abs(got - mean).max()
    assert int(flags.sum()) == 0
    del k, v
    torch.cuda.empty_cache()
