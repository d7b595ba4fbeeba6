"""Model-level prefill: a LLaMA / Qwen2 decoder stack whose attention is the
RIS hot path.

The paper replaces only the attention of the host model and leaves its
weights and every other layer as they are (Methods, opening of "The RIS
Implementation").  Per layer:

    ris_rmsnorm (fused residual add) -> QKV GEMM -> head-major V
    -> ris_rope_from on Q and K (head-major layout and rotation in one pass)
    -> ris_mask_build (this layer's geometry)
    -> ris_sparse_attn -> O GEMM -> ris_rmsnorm (fused residual add)
    -> gate/up GEMM -> ris_swiglu -> down GEMM

GEMMs are plain library GEMMs (torch.nn.functional.linear on the vendor
BLAS, weights kept [out, in] contiguous: activations times transposed
weights is the layout the library's bf16 GEMMs run fastest in, 13-16% ahead
of pre-transposed [in, out] weights at these shapes); every other step runs
in the library's kernels.  The stack
returns the final normalised hidden states (no LM head).
"""
import torch
import torch.nn.functional as F

from . import ris


class PrefillModel:
    """A decoder stack on one GPU.

    cfg: a model configuration with fields hidden, heads, kv_heads, head_dim,
    inter, layers, eps, qkv_bias, vocab.  weights: the dict layout of
    ``synth.model_weights`` (numpy arrays or tensors; linear weights
    [out, in]); they are copied to the device in ``dtype``.
    """

    def __init__(self, cfg, weights, device="cuda", dtype=torch.bfloat16):
        self.cfg = cfg
        self.dtype = dtype
        self.device = torch.device(device)

        def t(a):
            return torch.as_tensor(a).to(device=self.device, dtype=dtype).contiguous()

        self.embed = t(weights["embed"])
        self.layers = []
        for L in weights["layers"]:
            layer = {
                "wqkv": torch.cat([t(L["q"]), t(L["k"]), t(L["v"])], 0).contiguous(),   # [(Hq + 2 Hkv) D, hidden]
                "bqkv": torch.cat([t(L["bq"]), t(L["bk"]), t(L["bv"])]) if cfg.qkv_bias else None,
                "wo": t(L["o"]),                                                        # [hidden, Hq D]
                "wgu": torch.cat([t(L["gate"]), t(L["up"])], 0).contiguous(),          # [2 I, hidden]
                "wd": t(L["down"]),                                                     # [hidden, I]
                "ln1": t(L["ln1"]),
                "ln2": t(L["ln2"]),
            }
            self.layers.append(layer)
        self.norm = t(weights["norm"])
        self._csr = None

    def _csr_buffers(self, desc):
        cap = ris.mask_nnz_bound(desc)             # the bound does not depend on the layer
        rows = desc.heads * desc.N + 1
        if self._csr is None or self._csr[1].numel() < cap or self._csr[0].numel() != rows:
            self._csr = (torch.empty(rows, dtype=torch.int64, device=self.device),
                         torch.empty(max(cap, 1), dtype=torch.int32, device=self.device))
        return self._csr[0], self._csr[1], cap

    def attention(self, h, layer, l, mask, rope_desc, algo, timers=None):
        cfg = self.cfg
        N, D, Hq, Hkv = h.shape[0], cfg.head_dim, cfg.heads, cfg.kv_heads
        qkv = F.linear(h, layer["wqkv"], layer["bqkv"])
        v = qkv[:, (Hq + Hkv) * D:].view(N, Hkv, D).transpose(0, 1).contiguous()
        if timers:
            timers.mark("proj")
        # Q and K: head-major layout and rotation in one pass over the
        # projection output (ris_rope_from reads the strided head columns).
        qv = qkv[:, :Hq * D].view(N, Hq, D).transpose(0, 1)
        kv = qkv[:, Hq * D:(Hq + Hkv) * D].view(N, Hkv, D).transpose(0, 1)
        if rope_desc is not None:
            q = ris.rope_from(qv, torch.empty(Hq, N, D, dtype=qkv.dtype, device=qkv.device), rope_desc)
            k = ris.rope_from(kv, torch.empty(Hkv, N, D, dtype=qkv.dtype, device=qkv.device), rope_desc)
        else:
            q, k = qv.contiguous(), kv.contiguous()
        desc = ris.mask_desc(mask["mode"], mask["density_ppm"], N, Hkv, n_seeds=mask["n_seeds"],
                             seed=mask.get("seed", 0), layer=l, block=mask.get("block", 0),
                             window=mask.get("window", 0), anchor=mask.get("anchor", 0))
        row_ptr, col_idx, cap = self._csr_buffers(desc)
        if timers:
            timers.mark("rope")
        ris.mask_build(desc, row_ptr, col_idx, col_capacity=cap)
        if timers:
            timers.mark("geometry")
        out = torch.empty_like(q)
        ris.sparse_attn(q, k, v, row_ptr, col_idx, out,
                        ris.attn_desc(q, k, out, mode=mask["mode"], block=mask.get("block", 0), algo=algo))
        if timers:
            timers.mark("attention")
        a = out.transpose(0, 1).reshape(N, Hq * D)
        return F.linear(a, layer["wo"])

    def mlp(self, h, layer):
        gu = F.linear(h, layer["wgu"])
        m = torch.empty(h.shape[0], self.cfg.inter, dtype=self.dtype, device=self.device)
        ris.swiglu(gu, m)
        return F.linear(m, layer["wd"])

    def prefill(self, ids, mask, rope_desc=None, algo=ris.ATTN_AUTO, timers=None):
        """Final hidden states [N, hidden] for token ids (a device int64 tensor).

        mask: geometry parameters {mode, density_ppm, n_seeds[, seed, block,
        window, anchor]}; layer l uses layer index l.  rope_desc: from
        ``ris.rope_desc`` (None: no rotation).  timers: optional object with
        ``mark(name)`` called after each phase (for profiling).
        """
        cfg = self.cfg
        res = self.embed[ids].contiguous()                 # the residual stream
        h = torch.empty_like(res)
        ris.rmsnorm(res, self.layers[0]["ln1"], h, cfg.eps)
        for l, layer in enumerate(self.layers):
            a = self.attention(h, layer, l, mask, rope_desc, algo, timers)
            ris.rmsnorm(a, layer["ln2"], h, cfg.eps, residual=res)
            m = self.mlp(h, layer)
            nxt = self.layers[l + 1]["ln1"] if l + 1 < len(self.layers) else self.norm
            ris.rmsnorm(m, nxt, h, cfg.eps, residual=res)
            if timers:
                timers.mark("proj")
        return h
