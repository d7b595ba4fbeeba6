"""ris_decode_attn_static -- the decode step for callers that cannot allocate
(its partials live in the library's static per-GPU buffer) -- against
ris_decode_attn with a caller workspace, through the C ABI: bit-identical
outputs on two calls in a row, the second with a smaller batch (so the
static buffer holds the first call's partials when the second starts)."""
import pytest

from gpu_common import need_gpu, say, torch

pytestmark = pytest.mark.gpu


def decode_case(ris, B, seed, Hq=12, Hkv=2, D=128, N=6000, window=256, sink=4):
    """A batch of B sequences whose first generated token sat at N - 37 b,
    each decoding position t0 + 5: anchors built by the one-pass row build."""
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    max_len = N + 8
    t0s = [N - 37 * b for b in range(B)]
    Q = torch.randn(B, Hq, D, generator=gen, device="cuda").to(torch.bfloat16)
    K = torch.randn(B, Hkv, max_len, D, generator=gen, device="cuda").to(torch.bfloat16)
    V = torch.randn(B, Hkv, max_len, D, generator=gen, device="cuda").to(torch.bfloat16)
    md = ris.mask_desc(ris.STOCHASTIC, 10_000, max_len, Hkv, n_seeds=10, seed=seed)
    stride = max(ris.mask_rows_nnz_bound(md, t0, 1) for t0 in t0s)
    aptr = torch.zeros(B * (Hkv + 1), dtype=torch.int64, device="cuda")
    aidx = torch.zeros(B * stride, dtype=torch.int32, device="cuda")
    for b, t0 in enumerate(t0s):
        ris.mask_build_rows(md, t0, 1, aptr[b * (Hkv + 1):(b + 1) * (Hkv + 1)],
                            aidx[b * stride:(b + 1) * stride], col_capacity=stride)
    pos = torch.tensor([t0 + 5 for t0 in t0s], dtype=torch.int64, device="cuda")
    out = torch.empty(B, Hq, D, dtype=torch.float32, device="cuda")
    dd = ris.decode_desc(Q, K, out, stride, window=window, sink=sink)
    return Q, K, V, pos, aptr, aidx, out, dd


def test_static_decode_equals_workspace_decode():
    ris = need_gpu()
    for B, seed in [(24, 3), (5, 4)]:
        Q, K, V, pos, aptr, aidx, out, dd = decode_case(ris, B, seed)
        need = ris.decode_workspace_bytes(dd)
        say(f"static decode: batch {B}, partials {need} bytes of {ris.DECODE_STATIC_BYTES}")
        assert need <= ris.DECODE_STATIC_BYTES
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        ref = torch.empty_like(out)
        ris.decode_attn(Q, K, V, pos, aptr, aidx, ref, ws, dd)
        ris.decode_attn_static(Q, K, V, pos, aptr, aidx, out, dd)
        torch.cuda.synchronize()
        assert torch.isfinite(out).all()
        assert torch.equal(out, ref), float((out - ref).abs().max())
    with pytest.raises(ris.RisError) as e:
        big = ris.DecodeDesc(1, 0, 8000, 16, 2, 128, 16, 0, 16, 0, 0.0)
        ris.lib()
        import ctypes
        st = ris.lib().ris_decode_attn_static(None, None, None, None, None, None, None,
                                              ctypes.byref(big), None)
        ris._check(st, "ris_decode_attn_static")
    assert e.value.status == ris.E_CAPACITY
