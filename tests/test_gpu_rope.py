"""GPU RoPE (ris_rope) vs the oracle.

Tolerance, derived from the arithmetic the header states (float64 angle and
sincos, cos/sin rounded to float32, float32 rotation): each output is within
4 * 2^-24 * mscale * (|x_i| + |x_{i+D/2}|) of the exact rotation; a bf16
output adds one bf16 rounding (at most one bf16 ulp of the result).
"""
import numpy as np
import pytest

from gpu_common import bf16_ulp_tol, need_gpu, say, torch
from oracle import rope as o_rope
from synth import to_bf16

pytestmark = pytest.mark.gpu

CASES = [
    # kind, D, base, orig, factor, N, pos0, heads
    (o_rope.PLAIN, 128, 1e6, 32768, 0.0, 1000, 0, 3),
    (o_rope.PLAIN, 64, 1e4, 2048, 0.0, 333, 7, 2),
    (o_rope.LINEAR, 128, 1e6, 32768, 2.0, 512, 65000, 2),
    (o_rope.YARN, 128, 1e6, 32768, 0.0, 700, 64836, 2),    # factor from window = 2
    (o_rope.YARN, 64, 1e4, 2048, 32.0, 600, 64936, 4),     # TinyLlama at 32x
    (o_rope.YARN, 128, 1e6, 32768, 0.0, 500, 0, 1),        # window below native: s = 1
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", CASES)
def test_rope_matches_oracle(case, dtype):
    ris = need_gpu()
    kind, D, base, orig, factor, N, pos0, heads = case
    say(f"rope parity {case} {dtype}")
    rng = np.random.default_rng(D + N)
    x = rng.standard_normal((heads, N, D)).astype(np.float32)
    if dtype == "bf16":
        xt = to_bf16(x)
        x = xt.float().numpy()
    else:
        xt = torch.from_numpy(x)
    xd = xt.cuda()
    ris.rope(xd, ris.rope_desc(kind, base, orig_max_pos=orig, factor=factor), pos0=pos0)
    got = xd.float().cpu().numpy().astype(np.float64)

    s = o_rope.scale_factor(factor, pos0 + N, orig) if kind != o_rope.PLAIN else 1.0
    want = o_rope.apply(x, kind, base, pos0, s, orig)
    ms = o_rope.mscale(kind, s)
    pair = np.abs(x[..., : D // 2]) + np.abs(x[..., D // 2:])
    tol = 4 * 2.0**-24 * ms * np.concatenate([pair, pair], axis=-1) + 1e-30
    if dtype == "bf16":
        tol = tol + bf16_ulp_tol(want)
    err = np.abs(got - want)
    assert np.all(err <= tol), float((err - tol).max())


def test_rope_in_place_on_long_sequence_bf16():
    """Positions up to 65,535 with YaRN s = 2 (the 64k workload's setting)."""
    ris = need_gpu()
    heads, N, D = 2, 65536, 128
    rng = np.random.default_rng(11)
    xt = to_bf16(rng.standard_normal((heads, N, D)).astype(np.float32))
    xd = xt.cuda()
    ris.rope(xd, ris.rope_desc(ris.ROPE_YARN, 1e6, orig_max_pos=32768))
    got = xd.float().cpu().numpy()
    x = xt.float().numpy()
    rows = np.r_[0:64, N - 64:N]
    want = o_rope.apply(x[:, rows], o_rope.YARN, 1e6, s=2.0, orig_max_pos=32768, positions=rows)
    tol = bf16_ulp_tol(want) + 1e-5
    assert np.all(np.abs(got[:, rows] - want) <= tol)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_rope_from_strided_source(dtype):
    """ris_rope_from: the head columns of a token-major [N, (Hq + 2 Hkv) D]
    projection output, rotated into a contiguous [H, N, D] buffer, equal
    (bit for bit) ris_rope on a contiguous copy; the source is left as it was."""
    ris = need_gpu()
    Hq, Hkv, N, D = 6, 2, 777, 128
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    qkv = torch.randn(N, (Hq + 2 * Hkv) * D, generator=g, device="cuda").to(dtype)
    before = qkv.clone()
    rd = ris.rope_desc(ris.ROPE_YARN, 1e6, orig_max_pos=32768, factor=2.0)
    for lo, H in ((0, Hq), (Hq * D, Hkv)):
        view = qkv[:, lo:lo + H * D].view(N, H, D).transpose(0, 1)
        out = torch.empty(H, N, D, dtype=dtype, device="cuda")
        ris.rope_from(view, out, rd, pos0=64000)
        ref = view.contiguous()
        ris.rope(ref, rd, pos0=64000)
        torch.cuda.synchronize()
        assert torch.equal(out, ref)
    assert torch.equal(qkv, before)
