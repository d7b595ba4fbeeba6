"""Python binding of libris.so (ctypes).

Argument marshalling only: every step runs in the HIP library.  Tensors are
torch tensors used as device memory; streams are torch's current HIP stream
unless one is given.  A missing library raises -- there is no fallback.
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libris.so")

OK, E_ARG, E_SHAPE, E_DTYPE, E_CAPACITY, E_UNSUPPORTED, E_HIP, E_INCOMPLETE = 0, -1, -2, -3, -4, -5, -6, -7
STOCHASTIC, STRUCTURAL = 0, 1
F32, BF16 = 0, 1
ROPE_PLAIN, ROPE_LINEAR, ROPE_YARN = 0, 1, 2
ATTN_AUTO, ATTN_GATHER, ATTN_TILE = 0, 1, 2
MAX_N = 262144


class RisError(RuntimeError):
    def __init__(self, status, what):
        super().__init__(f"{what}: {status_string(status)} ({status})")
        self.status = status


class MaskDesc(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("density_ppm", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("n_seeds", ctypes.c_int32),
                ("layer", ctypes.c_int32), ("N", ctypes.c_int64), ("heads", ctypes.c_int32),
                ("causal", ctypes.c_int32), ("block", ctypes.c_int32),
                ("window", ctypes.c_int32), ("anchor", ctypes.c_int32)]


class RopeDesc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("base", ctypes.c_double),
                ("orig_max_pos", ctypes.c_int64), ("factor", ctypes.c_double),
                ("beta_slow", ctypes.c_double), ("beta_fast", ctypes.c_double)]


class AttnDesc(ctypes.Structure):
    _fields_ = [("dtype_in", ctypes.c_int32), ("dtype_out", ctypes.c_int32),
                ("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32), ("N", ctypes.c_int64),
                ("D", ctypes.c_int32), ("scale", ctypes.c_float), ("mode", ctypes.c_int32),
                ("block", ctypes.c_int32), ("causal", ctypes.c_int32), ("algo", ctypes.c_int32)]


class DecodeDesc(ctypes.Structure):
    _fields_ = [("dtype_in", ctypes.c_int32), ("dtype_out", ctypes.c_int32),
                ("batch", ctypes.c_int32), ("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32),
                ("D", ctypes.c_int32), ("max_len", ctypes.c_int64),
                ("anchor_stride", ctypes.c_int64), ("window", ctypes.c_int32),
                ("sink", ctypes.c_int32), ("scale", ctypes.c_float)]


_lib = None


def lib():
    """Load libris.so once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.ris_mask_build.argtypes = [ctypes.POINTER(MaskDesc), vp, vp, i64, vp]
        L.ris_mask_build.restype = ctypes.c_int
        L.ris_mask_nnz_bound.argtypes = [ctypes.POINTER(MaskDesc)]
        L.ris_mask_nnz_bound.restype = i64
        L.ris_mask_build_rows.argtypes = [ctypes.POINTER(MaskDesc), i64, i64, vp, vp, i64, vp]
        L.ris_mask_build_rows.restype = ctypes.c_int
        L.ris_mask_rows_nnz_bound.argtypes = [ctypes.POINTER(MaskDesc), i64, i64]
        L.ris_mask_rows_nnz_bound.restype = i64
        L.ris_rmsnorm.argtypes = [vp, vp, vp, vp, i64, i64, ctypes.c_float, i32, vp]
        L.ris_rmsnorm.restype = ctypes.c_int
        L.ris_swiglu.argtypes = [vp, vp, i64, i64, i32, vp]
        L.ris_swiglu.restype = ctypes.c_int
        L.ris_decode_workspace_bytes.argtypes = [ctypes.POINTER(DecodeDesc)]
        L.ris_decode_workspace_bytes.restype = i64
        L.ris_decode_attn.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i64,
                                      ctypes.POINTER(DecodeDesc), vp]
        L.ris_decode_attn.restype = ctypes.c_int
        L.ris_decode_attn_static.argtypes = [vp, vp, vp, vp, vp, vp, vp, ctypes.POINTER(DecodeDesc), vp]
        L.ris_decode_attn_static.restype = ctypes.c_int
        L.ris_rope.argtypes = [vp, i32, i32, i64, i32, i64, ctypes.POINTER(RopeDesc), vp]
        L.ris_rope.restype = ctypes.c_int
        L.ris_rope_from.argtypes = [vp, i64, i64, vp, i32, i32, i64, i32, i64, ctypes.POINTER(RopeDesc), vp]
        L.ris_rope_from.restype = ctypes.c_int
        L.ris_sparse_attn.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.POINTER(AttnDesc), vp]
        L.ris_sparse_attn.restype = ctypes.c_int
        L.ris_status_string.argtypes = [ctypes.c_int]
        L.ris_status_string.restype = ctypes.c_char_p
        L.ris_version.argtypes = []
        L.ris_version.restype = ctypes.c_int
        _lib = L
    return _lib


EXPORTS = ("ris_mask_build", "ris_mask_nnz_bound", "ris_mask_build_rows",
           "ris_mask_rows_nnz_bound", "ris_rope", "ris_rope_from", "ris_sparse_attn",
           "ris_decode_workspace_bytes", "ris_decode_attn", "ris_decode_attn_static", "ris_rmsnorm",
           "ris_swiglu",
           "ris_status_string", "ris_version")


def status_string(status):
    return lib().ris_status_string(int(status)).decode()


def version():
    return lib().ris_version()


def _check(status, what):
    if status != OK:
        raise RisError(status, what)


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(stream if isinstance(stream, int) else stream.cuda_stream)
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _need_device(*ts):
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError("tensors must be contiguous GPU tensors")


def _capacity(col_idx, col_capacity):
    """Entries the library may write: col_idx's size unless a smaller
    capacity is given.  A capacity beyond the tensor would let the kernel
    write past it, so it is refused here."""
    if col_idx is None:
        return 0
    if col_capacity is None:
        return col_idx.numel()
    if col_capacity < 0 or col_capacity > col_idx.numel():
        raise ValueError(f"col_capacity {col_capacity} outside [0, {col_idx.numel()}] (col_idx size)")
    return int(col_capacity)


def mask_desc(mode, density_ppm, N, heads, n_seeds=1, seed=0, layer=0, causal=1, block=0,
              window=0, anchor=0):
    return MaskDesc(mode, density_ppm, seed, n_seeds, layer, N, heads, causal, block, window,
                    anchor)


def mask_nnz_bound(desc):
    v = lib().ris_mask_nnz_bound(ctypes.byref(desc))
    if v < 0:
        raise RisError(int(v), "ris_mask_nnz_bound")
    return int(v)


def mask_build(desc, row_ptr, col_idx=None, col_capacity=None, stream=None):
    """ris_mask_build: count phase when col_idx is None, else fill phase."""
    import torch
    _need_device(row_ptr, col_idx)
    if row_ptr.dtype != torch.int64 or row_ptr.numel() != desc.heads * desc.N + 1:
        raise ValueError("row_ptr must be int64[heads*N + 1]")
    if col_idx is not None and col_idx.dtype != torch.int32:
        raise ValueError("col_idx must be int32")
    cap = _capacity(col_idx, col_capacity)
    _check(lib().ris_mask_build(ctypes.byref(desc), _ptr(row_ptr), _ptr(col_idx), cap,
                                _stream(stream)), "ris_mask_build")


def mask_rows_nnz_bound(desc, q_begin, q_count):
    v = lib().ris_mask_rows_nnz_bound(ctypes.byref(desc), q_begin, q_count)
    if v < 0:
        raise RisError(int(v), "ris_mask_rows_nnz_bound")
    return int(v)


def mask_build_rows(desc, q_begin, q_count, row_ptr, col_idx=None, col_capacity=None,
                    stream=None):
    """ris_mask_build_rows: rows [q_begin, q_begin + q_count) of every head.
    row_ptr and col_idx may be views into larger buffers (e.g. one sequence's
    slice of a batched anchor cache)."""
    import torch
    if row_ptr.dtype != torch.int64 or row_ptr.numel() != desc.heads * q_count + 1:
        raise ValueError("row_ptr must be int64[heads*q_count + 1]")
    if not row_ptr.is_cuda or row_ptr.stride(0) != 1:
        raise ValueError("row_ptr must be a dense GPU vector")
    if col_idx is not None and (col_idx.dtype != torch.int32 or not col_idx.is_cuda
                                or col_idx.stride(0) != 1):
        raise ValueError("col_idx must be a dense int32 GPU vector")
    cap = _capacity(col_idx, col_capacity)
    _check(lib().ris_mask_build_rows(ctypes.byref(desc), q_begin, q_count, _ptr(row_ptr),
                                     _ptr(col_idx), cap, _stream(stream)), "ris_mask_build_rows")


def decode_desc(Q, K, out, anchor_stride, window=0, sink=0, scale=0.0):
    """Descriptor from Q [B, Hq, D], the cache K [B, Hkv, max_len, D] and out."""
    B, Hq, D = Q.shape
    return DecodeDesc(_dtype_code(Q), _dtype_code(out), B, Hq, K.shape[1], D, K.shape[2],
                      anchor_stride, window, sink, scale)


def decode_workspace_bytes(desc):
    v = lib().ris_decode_workspace_bytes(ctypes.byref(desc))
    if v < 0:
        raise RisError(int(v), "ris_decode_workspace_bytes")
    return int(v)


def decode_attn(Q, K, V, pos, anchor_ptr, anchor_idx, out, workspace, desc, stream=None):
    """ris_decode_attn; workspace is a device uint8 tensor of at least
    decode_workspace_bytes(desc) bytes."""
    import torch
    _need_device(Q, K, V, pos, anchor_ptr, anchor_idx, out, workspace)
    if pos.dtype != torch.int64 or anchor_ptr.dtype != torch.int64:
        raise TypeError("pos and anchor_ptr must be int64")
    if anchor_idx.dtype != torch.int32:
        raise TypeError("anchor_idx must be int32")
    if pos.numel() != desc.batch or anchor_ptr.numel() != desc.batch * (desc.Hkv + 1):
        raise ValueError("pos must hold B entries and anchor_ptr B * (Hkv + 1)")
    if anchor_idx.numel() < desc.batch * desc.anchor_stride:
        raise ValueError("anchor_idx must hold B * anchor_stride entries")
    if not (Q.dtype == K.dtype == V.dtype) or K.shape != V.shape:
        raise TypeError("Q, K, V must share a dtype and K, V a shape")
    if _dtype_code(Q) != desc.dtype_in or _dtype_code(out) != desc.dtype_out:
        raise TypeError("Q and out dtypes must match the descriptor")
    if (tuple(Q.shape) != (desc.batch, desc.Hq, desc.D) or tuple(out.shape) != tuple(Q.shape)
            or tuple(K.shape) != (desc.batch, desc.Hkv, desc.max_len, desc.D)):
        raise ValueError("Q and out must be [B, Hq, D] and K, V [B, Hkv, max_len, D] as in the descriptor")
    nbytes = workspace.numel() * workspace.element_size()
    _check(lib().ris_decode_attn(_ptr(Q), _ptr(K), _ptr(V), _ptr(pos), _ptr(anchor_ptr),
                                 _ptr(anchor_idx), _ptr(out), _ptr(workspace), nbytes,
                                 ctypes.byref(desc), _stream(stream)), "ris_decode_attn")
    return out


DECODE_STATIC_BYTES = 32 << 20


def decode_attn_static(Q, K, V, pos, anchor_ptr, anchor_idx, out, desc, stream=None):
    """ris_decode_attn_static: the decode step with the library's static
    per-GPU partials (no workspace; nothing is allocated).  Calls that may
    overlap on one GPU race on that buffer."""
    import torch
    _need_device(Q, K, V, pos, anchor_ptr, anchor_idx, out)
    if pos.dtype != torch.int64 or anchor_ptr.dtype != torch.int64 or anchor_idx.dtype != torch.int32:
        raise TypeError("pos and anchor_ptr must be int64, anchor_idx int32")
    if pos.numel() != desc.batch or anchor_ptr.numel() != desc.batch * (desc.Hkv + 1):
        raise ValueError("pos must hold B entries and anchor_ptr B * (Hkv + 1)")
    if anchor_idx.numel() < desc.batch * desc.anchor_stride:
        raise ValueError("anchor_idx must hold B * anchor_stride entries")
    if not (Q.dtype == K.dtype == V.dtype) or K.shape != V.shape:
        raise TypeError("Q, K, V must share a dtype and K, V a shape")
    if _dtype_code(Q) != desc.dtype_in or _dtype_code(out) != desc.dtype_out:
        raise TypeError("Q and out dtypes must match the descriptor")
    if (tuple(Q.shape) != (desc.batch, desc.Hq, desc.D) or tuple(out.shape) != tuple(Q.shape)
            or tuple(K.shape) != (desc.batch, desc.Hkv, desc.max_len, desc.D)):
        raise ValueError("Q and out must be [B, Hq, D] and K, V [B, Hkv, max_len, D] as in the descriptor")
    _check(lib().ris_decode_attn_static(_ptr(Q), _ptr(K), _ptr(V), _ptr(pos), _ptr(anchor_ptr),
                                        _ptr(anchor_idx), _ptr(out), ctypes.byref(desc), _stream(stream)),
           "ris_decode_attn_static")
    return out


def rmsnorm(x, weight, out, eps, residual=None, stream=None):
    """ris_rmsnorm over the last dimension of x (rows = everything else)."""
    _need_device(x, weight, out, residual)
    cols = x.shape[-1]
    if weight.numel() != cols or out.shape != x.shape or (residual is not None and residual.shape != x.shape):
        raise ValueError("shapes: weight [cols], out and residual like x")
    if not (x.dtype == weight.dtype == out.dtype) or (residual is not None and residual.dtype != x.dtype):
        raise TypeError("x, weight, out (and residual) must share a dtype")
    _check(lib().ris_rmsnorm(_ptr(x), _ptr(residual), _ptr(weight), _ptr(out), x.numel() // cols, cols,
                             eps, _dtype_code(x), _stream(stream)), "ris_rmsnorm")
    return out


def swiglu(gate_up, out, stream=None):
    """ris_swiglu: out [rows, I] from gate_up [rows, 2I]."""
    _need_device(gate_up, out)
    inter = out.shape[-1]
    if gate_up.shape[-1] != 2 * inter or gate_up.numel() != 2 * out.numel() or gate_up.dtype != out.dtype:
        raise ValueError("gate_up must be [rows, 2*inter] of out's dtype")
    _check(lib().ris_swiglu(_ptr(gate_up), _ptr(out), out.numel() // inter, inter, _dtype_code(out),
                            _stream(stream)), "ris_swiglu")
    return out


def rope(x, desc, pos0=0, stream=None):
    """ris_rope on x [heads, N, D] in place."""
    _need_device(x)
    H, N, D = x.shape
    _check(lib().ris_rope(_ptr(x), _dtype_code(x), H, N, D, pos0, ctypes.byref(desc),
                          _stream(stream)), "ris_rope")
    return x


def rope_from(src, out, desc, pos0=0, stream=None):
    """ris_rope_from: src is a [heads, N, D] view (any head and token strides,
    unit stride along D, e.g. a head-column view of a token-major projection
    output); out is [heads, N, D] contiguous and receives the rotated rows."""
    _need_device(out)
    H, N, D = out.shape
    if (not src.is_cuda or src.device != out.device or tuple(src.shape) != (H, N, D) or src.stride(2) != 1
            or src.dtype != out.dtype):
        raise ValueError("src must be a [heads, N, D] device view of out's dtype with unit stride along D")
    _check(lib().ris_rope_from(_ptr(src), src.stride(0), src.stride(1), _ptr(out), _dtype_code(out), H, N, D,
                               pos0, ctypes.byref(desc), _stream(stream)), "ris_rope_from")
    return out


def rope_desc(kind, base, orig_max_pos=0, factor=0.0, beta_slow=0.0, beta_fast=0.0):
    return RopeDesc(kind, base, orig_max_pos, factor, beta_slow, beta_fast)


def attn_desc(Q, K, out, mode=STOCHASTIC, block=0, causal=1, scale=0.0, algo=ATTN_AUTO):
    Hq, N, D = Q.shape
    return AttnDesc(_dtype_code(Q), _dtype_code(out), Hq, K.shape[0], N, D, scale, mode,
                    block, causal, algo)


def sparse_attn(Q, K, V, row_ptr, col_idx, out, desc, stream=None):
    """ris_sparse_attn: out[Hq, N, D] from the CSR sets.  The tensors are
    checked against the descriptor before anything is launched."""
    import torch
    _need_device(Q, K, V, row_ptr, col_idx, out)
    if not (Q.dtype == K.dtype == V.dtype):
        raise TypeError("Q, K, V must share a dtype")
    if _dtype_code(Q) != desc.dtype_in or _dtype_code(out) != desc.dtype_out:
        raise TypeError("Q and out dtypes must match the descriptor")
    q_shape, kv_shape = (desc.Hq, desc.N, desc.D), (desc.Hkv, desc.N, desc.D)
    if tuple(Q.shape) != q_shape or tuple(out.shape) != q_shape or tuple(K.shape) != kv_shape \
            or tuple(V.shape) != kv_shape:
        raise ValueError(f"Q and out must be {q_shape}, K and V {kv_shape}")
    if row_ptr.dtype != torch.int64 or row_ptr.numel() != desc.Hkv * desc.N + 1 or col_idx.dtype != torch.int32:
        raise ValueError("row_ptr must be int64[Hkv*N + 1] and col_idx int32")
    if len({t.device for t in (Q, K, V, row_ptr, col_idx, out)}) != 1:
        raise ValueError("all tensors must be on one device")
    _check(lib().ris_sparse_attn(_ptr(Q), _ptr(K), _ptr(V), _ptr(row_ptr), _ptr(col_idx),
                                 _ptr(out), ctypes.byref(desc), _stream(stream)),
           "ris_sparse_attn")
    return out


def check_complete(row_ptr, stream=None):
    """Read row_ptr's total back (one 8-byte copy, after the work queued on
    `stream`) and raise RisError(E_INCOMPLETE) when the one-pass build
    reported an incomplete CSR (a negative total); returns nnz."""
    import torch
    if stream is not None:
        torch.cuda.synchronize(row_ptr.device)
    nnz = int(row_ptr[-1].item())
    if nnz < 0:
        raise RisError(E_INCOMPLETE, "ris_mask_build")
    return nnz


def build_csr(desc, device="cuda", stream=None, use_bound=False):
    """Both phases of ris_mask_build; returns (row_ptr, col_idx) on the device.

    use_bound sizes col_idx from the host-side bound (one pass, then one
    8-byte read-back of the total to check that the build is complete);
    otherwise the exact nnz is read back between the count and fill phases.
    """
    import torch
    row_ptr = torch.empty(desc.heads * desc.N + 1, dtype=torch.int64, device=device)
    if use_bound:
        # Bound-sized col_idx: one fused call computes row_ptr and col_idx.
        cap = mask_nnz_bound(desc)
    else:
        mask_build(desc, row_ptr, None, stream=stream)
        if stream is not None:
            # The read-back below runs on torch's current stream; the count
            # ran on the caller's, so wait for the device first.
            torch.cuda.synchronize(row_ptr.device)
        cap = int(row_ptr[-1].item())
    col_idx = torch.empty(max(cap, 1), dtype=torch.int32, device=device)
    mask_build(desc, row_ptr, col_idx, col_capacity=cap, stream=stream)
    if use_bound:
        check_complete(row_ptr, stream)
    return row_ptr, col_idx
