"""Thin Python binding of libbt (ctypes).

Argument marshalling only: every computation runs in the HIP kernels of
libbt.so.  PyTorch supplies device memory (tensors) and the current HIP
stream.  Function names mirror the C ABI declared in include/bt.h.

Importing this module does not load the library; the first call does, and
raises BTLibraryError if libbt.so has not been built -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbt.so")

OP_N, OP_T = 0, 1
EPI_NONE, EPI_BIAS, EPI_BIAS_GELU, EPI_DGELU = 0, 1, 2, 3

_c = ctypes
vp = _c.c_void_p
i32 = _c.c_int
f32 = _c.c_float
sz = _c.c_size_t


class BTLibraryError(RuntimeError):
    pass


class BTError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


class BTNonFiniteError(BTError):
    """A training step met a non-finite gradient norm and skipped its update."""


BT_ENONFINITE = 6


PROF_CLASSES = ("gemm", "attn_fwd", "attn_bwd", "ln_fwd", "ln_bwd", "xent", "emb_fwd", "emb_bwd",
                "colsum", "grad_norm", "adamw", "other")


class KernelStat(_c.Structure):
    _fields_ = [("launches", _c.c_longlong), ("ms", _c.c_double), ("flops", _c.c_double),
                ("bytes", _c.c_double)]


f64 = _c.c_double


class GPT2ConfigC(_c.Structure):
    _fields_ = [("V", i32), ("Vp", i32), ("max_T", i32), ("L", i32), ("H", i32), ("C", i32),
                ("ln_eps", f32), ("lr", f64), ("beta1", f64), ("beta2", f64), ("adam_eps", f64),
                ("weight_decay", f64), ("grad_clip", f64)]


class CPSegments(_c.Structure):
    """bt_cp_segments: a rank's query rows and a shard's key/value rows as 1 or
    2 segments of `seg` tokens starting at global positions q_pos / k_pos."""
    _fields_ = [("seg", i32), ("n_q", i32), ("n_k", i32), ("q_pos", i32 * 2), ("k_pos", i32 * 2)]


def cp_segments(seg, q_pos, k_pos) -> CPSegments:
    """Build a CPSegments from position lists (1 or 2 entries per side)."""
    g = CPSegments()
    g.seg, g.n_q, g.n_k = seg, len(q_pos), len(k_pos)
    for i, v in enumerate(q_pos):
        g.q_pos[i] = v
    for i, v in enumerate(k_pos):
        g.k_pos[i] = v
    return g


i64 = _c.c_longlong

_SIGS = {
    "bt_status_str": (_c.c_char_p, [i32]),
    "bt_last_error": (_c.c_char_p, []),
    "bt_last_status": (i32, []),
    "bt_version": (_c.c_char_p, []),
    "bt_gemm": (i32, [i32, i32, i32, i32, i32, vp, i32, vp, i32, f32, vp, i32, vp, i32, vp, vp, vp, vp, vp, sz, vp]),
    "bt_gemm_ws_bytes": (sz, [i32, i32, i32, i32, i32, i32]),
    "bt_gemm_plan": (i32, [i32, i32, i32, i32, i32, i32, i32, _c.POINTER(i32), _c.POINTER(i32), _c.POINTER(i32)]),
    "bt_gemm_noalloc": (i32, [i32, i32, i32, i32, i32, vp, i32, vp, i32, f32, vp, i32, vp, i32, vp, vp, vp, vp, vp]),
    "bt_gemm_noalloc_max_ws_bytes": (sz, []),
    "bt_attention_fwd": (i32, [vp, vp, vp, i32, i32, i32, i32, vp]),
    "bt_attention_bwd": (i32, [vp, vp, vp, vp, vp, vp, sz, i32, i32, i32, i32, vp]),
    "bt_attention_bwd_ws_bytes": (sz, [i32, i32, i32, i32]),
    "bt_attention_bwd_ws_min_bytes": (sz, [i32, i32, i32, i32]),
    "bt_cp_rank_segments": (i32, [i32, i32, i32, i32, _c.POINTER(CPSegments)]),
    "bt_cp_shard_tokens": (i32, [vp, vp, i32, i32, i32, i32, vp]),
    "bt_attention_block_fwd": (i32, [vp, vp, i64, vp, vp, i32, i32, i32, i32, _c.POINTER(CPSegments), vp]),
    "bt_attention_lse_merge": (i32, [vp, vp, vp, vp, i32, i32, i32, i32, vp]),
    "bt_attention_rowdot": (i32, [vp, vp, vp, i32, i32, i32, i32, vp]),
    "bt_attention_block_bwd": (i32, [vp, vp, vp, i64, vp, vp, vp, vp, i32, vp, sz, i32, i32, i32,
                                     _c.POINTER(CPSegments), vp]),
    "bt_attention_block_bwd_ws_bytes": (sz, [i32, i32, i32, _c.POINTER(CPSegments)]),
    "bt_layernorm_fwd": (i32, [vp, vp, vp, vp, vp, vp, i32, i32, f32, vp]),
    "bt_layernorm_bwd": (i32, [vp, vp, vp, vp, vp, vp, vp, vp, f32, f32, vp, sz, i32, i32, vp]),
    "bt_layernorm_bwd_ws_bytes": (sz, [i32, i32]),
    "bt_gelu_fwd": (i32, [vp, vp, sz, vp]),
    "bt_gelu_bwd": (i32, [vp, vp, vp, sz, vp]),
    "bt_softmax_xent_fwd": (i32, [vp, vp, vp, vp, i32, i32, i32, vp]),
    "bt_softmax_xent_bwd": (i32, [vp, vp, vp, vp, f32, i32, i32, i32, vp]),
    "bt_softmax_xent_fused": (i32, [vp, vp, vp, vp, f32, i32, i32, i32, vp]),
    "bt_adamw_step": (i32, [vp, vp, vp, vp, sz, sz, _c.c_double, _c.c_double, _c.c_double, _c.c_double,
                            _c.c_double, i32, vp, vp]),
    "bt_grad_norm_clip": (i32, [vp, sz, f32, vp, vp, vp, sz, vp]),
    "bt_grad_norm_ws_bytes": (sz, [sz]),
    "bt_embedding_fwd": (i32, [vp, vp, vp, vp, i32, i32, i32, i32, vp]),
    "bt_embedding_bwd": (i32, [vp, vp, vp, vp, f32, vp, sz, i32, i32, i32, i32, vp]),
    "bt_embedding_bwd_ws_bytes": (sz, [i32, i32, i32, i32]),
    "bt_embedding_index_bytes": (sz, [i32, i32]),
    "bt_embedding_index": (i32, [vp, vp, sz, i32, i32, i32, vp]),
    "bt_embedding_bwd_indexed": (i32, [vp, sz, vp, vp, vp, f32, vp, sz, i32, i32, i32, i32, vp]),
    "bt_embedding_bwd_indexed_ws_bytes": (sz, [i32, i32, i32]),
    "bt_colsum": (i32, [vp, i32, i32, i32, vp, f32, vp, sz, vp]),
    "bt_colsum_ws_bytes": (sz, [i32, i32]),
    "bt_gpt2_num_params": (sz, [_c.POINTER(GPT2ConfigC)]),
    "bt_gpt2_num_decay_params": (sz, [_c.POINTER(GPT2ConfigC)]),
    "bt_gpt2_param_offsets": (i32, [_c.POINTER(GPT2ConfigC), _c.POINTER(sz), _c.POINTER(i32)]),
    "bt_gpt2_workspace_bytes": (sz, [_c.POINTER(GPT2ConfigC), i32, i32]),
    "bt_gpt2_create": (i32, [_c.POINTER(GPT2ConfigC), vp, sz, i32, i32, vp, _c.POINTER(vp)]),
    "bt_gpt2_destroy": (None, [vp]),
    "bt_gpt2_step_count": (i32, [vp]),
    "bt_gpt2_set_step_count": (None, [vp, i32]),
    "bt_gpt2_read_scalars": (i32, [vp, _c.POINTER(f32)]),
    "bt_gpt2_fwd_bwd": (i32, [vp, vp, vp, vp, vp, i32, i32, f32, i32, vp, vp]),
    "bt_gpt2_optimizer_step": (i32, [vp, vp, vp, vp, i32, _c.c_double]),
    "bt_gpt2_train_step": (f32, [vp, vp, vp, vp, vp, vp, i32, i32]),
    "bt_gpt2_profile_enable": (i32, [vp, i32]),
    "bt_gpt2_profile_read": (i32, [vp, _c.POINTER(KernelStat), i32]),
}

EXPORTED = tuple(_SIGS)

_lib = None


def lib():
    """Load libbt.so (once).  Raises BTLibraryError if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise BTLibraryError(
                f"{LIB_PATH} is not built; run `python -m paper_2606_24780_amd.build` first")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status: int, where: str):
    if status != 0:
        L = lib()
        raise BTError(status, where, f"{L.bt_status_str(status).decode()}: {L.bt_last_error().decode()}")


def _torch():
    import torch
    return torch


def _p(t) -> Optional[int]:
    """Device pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    return t.data_ptr()


def _f32(t, name):
    torch = _torch()
    if t is not None and (t.dtype != torch.float32 or not t.is_cuda):
        raise TypeError(f"{name} must be a float32 GPU tensor")
    return t


def _stream(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _ws(nbytes: int, ws=None, device=None):
    torch = _torch()
    if nbytes == 0:
        return None
    if ws is not None:
        return ws
    return torch.empty(nbytes, dtype=torch.uint8, device=device or "cuda")


# ---------------------------------------------------------------- operations
def bt_gemm(opA, opB, M, N, K, A, lda, B, ldb, beta, C, ldc, bias=None, epi=EPI_NONE,
            preact_out=None, gelu_in=None, residual=None, colsum_B=None, ws=None, stream=None):
    L = lib()
    need = L.bt_gemm_ws_bytes(opA, opB, M, N, K, epi)
    w = _ws(need, ws, C.device)
    nbytes = 0 if w is None else w.numel() * w.element_size()
    _check(L.bt_gemm(opA, opB, M, N, K, _p(A), lda, _p(B), ldb, beta, _p(C), ldc, _p(bias), epi,
                     _p(preact_out), _p(gelu_in), _p(residual), _p(colsum_B), _p(w), nbytes,
                     _stream(stream)), "bt_gemm")
    return C


def bt_gemm_plan(opA, opB, M, N, K, lda, ldb):
    """(tile_depth, splits, direct) of the launch bt_gemm makes for the product."""
    d, sp, dr = i32(0), i32(0), i32(0)
    _check(lib().bt_gemm_plan(opA, opB, M, N, K, lda, ldb, _c.byref(d), _c.byref(sp), _c.byref(dr)),
           "bt_gemm_plan")
    return d.value, sp.value, dr.value


def bt_gemm_noalloc(opA, opB, M, N, K, A, lda, B, ldb, beta, C, ldc, bias=None, epi=EPI_NONE,
                    preact_out=None, gelu_in=None, residual=None, colsum_B=None, stream=None):
    """bt_gemm with the library's static split-K scratch: allocates nothing."""
    _check(lib().bt_gemm_noalloc(opA, opB, M, N, K, _p(A), lda, _p(B), ldb, beta, _p(C), ldc, _p(bias), epi,
                                 _p(preact_out), _p(gelu_in), _p(residual), _p(colsum_B), _stream(stream)),
           "bt_gemm_noalloc")
    return C


def bt_attention_fwd(qkv, out, lse, B, T, H, hd, stream=None):
    _check(lib().bt_attention_fwd(_p(qkv), _p(out), _p(lse), B, T, H, hd, _stream(stream)),
           "bt_attention_fwd")


def bt_attention_bwd(dout, qkv, out, lse, dqkv, B, T, H, hd, ws=None, stream=None, small_ws=False):
    """small_ws: allocate only bt_attention_bwd_ws_min_bytes (the method that
    recomputes S and dP for dQ instead of storing dS)."""
    L = lib()
    need = (L.bt_attention_bwd_ws_min_bytes if small_ws else L.bt_attention_bwd_ws_bytes)(B, T, H, hd)
    w = _ws(need, ws, qkv.device)
    _check(L.bt_attention_bwd(_p(dout), _p(qkv), _p(out), _p(lse), _p(dqkv), _p(w),
                              0 if w is None else w.numel() * w.element_size(), B, T, H, hd,
                              _stream(stream)), "bt_attention_bwd")


def bt_cp_rank_segments(T, W, rank, shard) -> CPSegments:
    g = CPSegments()
    _check(lib().bt_cp_rank_segments(T, W, rank, shard, _c.byref(g)), "bt_cp_rank_segments")
    return g


def bt_cp_shard_tokens(tokens, local, B, T, W, rank, stream=None):
    _check(lib().bt_cp_shard_tokens(_p(tokens), _p(local), B, T, W, rank, _stream(stream)),
           "bt_cp_shard_tokens")


def bt_attention_block_fwd(qkv, kv, kv_stride, out, lse, merge, B, H, hd, segs, stream=None):
    _check(lib().bt_attention_block_fwd(_p(qkv), _p(kv), kv_stride, _p(out), _p(lse), int(merge), B, H, hd,
                                        _c.byref(segs), _stream(stream)), "bt_attention_block_fwd")


def bt_attention_lse_merge(out, lse, block_out, block_lse, B, T, H, hd, stream=None):
    _check(lib().bt_attention_lse_merge(_p(out), _p(lse), _p(block_out), _p(block_lse), B, T, H, hd,
                                        _stream(stream)), "bt_attention_lse_merge")


def bt_attention_rowdot(dout, out, D, B, T, H, hd, stream=None):
    _check(lib().bt_attention_rowdot(_p(dout), _p(out), _p(D), B, T, H, hd, _stream(stream)),
           "bt_attention_rowdot")


def bt_attention_block_bwd(dout, qkv, kv, kv_stride, lse, D, dqkv, dkv, accumulate, B, H, hd, segs,
                           ws=None, stream=None):
    """ws: a uint8 tensor of at least bt_attention_block_bwd_ws_bytes() selects
    the stored-dS method; None, the recomputing one."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().bt_attention_block_bwd(_p(dout), _p(qkv), _p(kv), kv_stride, _p(lse), _p(D), _p(dqkv),
                                        _p(dkv), int(accumulate), _p(ws), nbytes, B, H, hd, _c.byref(segs),
                                        _stream(stream)), "bt_attention_block_bwd")


def bt_attention_block_bwd_ws_bytes(B, H, hd, segs) -> int:
    return lib().bt_attention_block_bwd_ws_bytes(B, H, hd, _c.byref(segs))


def bt_layernorm_fwd(x, gamma, beta, y, mean, rstd, M, C, eps=1e-5, stream=None):
    _check(lib().bt_layernorm_fwd(_p(x), _p(gamma), _p(beta), _p(y), _p(mean), _p(rstd), M, C, eps,
                                  _stream(stream)), "bt_layernorm_fwd")


def bt_layernorm_bwd(dy, x, gamma, mean, rstd, dx, dgamma, dbeta, dx_beta, param_beta, M, C,
                     ws=None, stream=None):
    L = lib()
    w = _ws(L.bt_layernorm_bwd_ws_bytes(M, C), ws, x.device)
    _check(L.bt_layernorm_bwd(_p(dy), _p(x), _p(gamma), _p(mean), _p(rstd), _p(dx), _p(dgamma),
                              _p(dbeta), dx_beta, param_beta, _p(w),
                              0 if w is None else w.numel() * w.element_size(), M, C, _stream(stream)),
           "bt_layernorm_bwd")


def bt_gelu_fwd(x, y, n=None, stream=None):
    _check(lib().bt_gelu_fwd(_p(x), _p(y), x.numel() if n is None else n, _stream(stream)), "bt_gelu_fwd")


def bt_gelu_bwd(x, dy, dx, n=None, stream=None):
    _check(lib().bt_gelu_bwd(_p(x), _p(dy), _p(dx), x.numel() if n is None else n, _stream(stream)),
           "bt_gelu_bwd")


def bt_softmax_xent_fwd(logits, targets, loss_rows, lse, M, V, Vp, stream=None):
    _check(lib().bt_softmax_xent_fwd(_p(logits), _p(targets), _p(loss_rows), _p(lse), M, V, Vp,
                                     _stream(stream)), "bt_softmax_xent_fwd")


def bt_softmax_xent_bwd(logits, lse, targets, dlogits, scale, M, V, Vp, stream=None):
    _check(lib().bt_softmax_xent_bwd(_p(logits), _p(lse), _p(targets), _p(dlogits), scale, M, V, Vp,
                                     _stream(stream)), "bt_softmax_xent_bwd")


def bt_softmax_xent_fused(logits, targets, loss_rows, lse, scale, M, V, Vp, stream=None):
    _check(lib().bt_softmax_xent_fused(_p(logits), _p(targets), _p(loss_rows), _p(lse), scale, M, V, Vp,
                                       _stream(stream)), "bt_softmax_xent_fused")


def bt_adamw_step(p, g, m, v, n, n_decay, lr, beta1, beta2, eps, weight_decay, t, grad_scale=None,
                  stream=None):
    _check(lib().bt_adamw_step(_p(p), _p(g), _p(m), _p(v), n, n_decay, lr, beta1, beta2, eps,
                               weight_decay, t, _p(grad_scale), _stream(stream)), "bt_adamw_step")


def bt_grad_norm_clip(g, n, clip, out_norm, out_coef, ws=None, stream=None):
    L = lib()
    w = _ws(L.bt_grad_norm_ws_bytes(n), ws, g.device)
    _check(L.bt_grad_norm_clip(_p(g), n, clip, _p(out_norm), _p(out_coef), _p(w),
                               0 if w is None else w.numel() * w.element_size(), _stream(stream)),
           "bt_grad_norm_clip")


def bt_embedding_fwd(tokens, wte, wpe, x0, B, T, C, Vp, stream=None):
    _check(lib().bt_embedding_fwd(_p(tokens), _p(wte), _p(wpe), _p(x0), B, T, C, Vp, _stream(stream)),
           "bt_embedding_fwd")


def bt_embedding_bwd(tokens, dx0, dwte, dwpe, wpe_beta, B, T, C, Vp, ws=None, stream=None):
    L = lib()
    w = _ws(L.bt_embedding_bwd_ws_bytes(B, T, C, Vp), ws, dx0.device)
    _check(L.bt_embedding_bwd(_p(tokens), _p(dx0), _p(dwte), _p(dwpe), wpe_beta, _p(w),
                              0 if w is None else w.numel() * w.element_size(), B, T, C, Vp,
                              _stream(stream)), "bt_embedding_bwd")


def bt_embedding_index(tokens, index, B, T, Vp, stream=None):
    """index: a uint8 GPU tensor of at least bt_embedding_index_bytes(B, T) bytes."""
    _check(lib().bt_embedding_index(_p(tokens), _p(index), index.numel(), B, T, Vp, _stream(stream)),
           "bt_embedding_index")


def bt_embedding_bwd_indexed(index, dx0, dwte, dwpe, wpe_beta, B, T, C, Vp, ws=None, stream=None):
    L = lib()
    w = _ws(L.bt_embedding_bwd_indexed_ws_bytes(B, T, C), ws, dx0.device)
    _check(L.bt_embedding_bwd_indexed(_p(index), index.numel(), _p(dx0), _p(dwte), _p(dwpe), wpe_beta, _p(w),
                                      0 if w is None else w.numel() * w.element_size(), B, T, C, Vp,
                                      _stream(stream)), "bt_embedding_bwd_indexed")


def bt_colsum(X, M, N, ldx, out, beta, ws=None, stream=None):
    L = lib()
    w = _ws(L.bt_colsum_ws_bytes(M, N), ws, out.device)
    _check(L.bt_colsum(_p(X), M, N, ldx, _p(out), beta, _p(w),
                       0 if w is None else w.numel() * w.element_size(), _stream(stream)), "bt_colsum")


# -------------------------------------------------------------- composed step
def make_config(cfg, hp) -> GPT2ConfigC:
    return GPT2ConfigC(cfg.V, cfg.Vp, cfg.max_T, cfg.L, cfg.H, cfg.C, cfg.ln_eps, hp.lr, hp.beta1,
                       hp.beta2, hp.eps, hp.weight_decay, hp.grad_clip)


def num_params(cfg, hp) -> int:
    return lib().bt_gpt2_num_params(_c.byref(make_config(cfg, hp)))


def param_offsets(cfg, hp):
    L = lib()
    c = make_config(cfg, hp)
    n = i32(0)
    _check(L.bt_gpt2_param_offsets(_c.byref(c), None, _c.byref(n)), "bt_gpt2_param_offsets")
    arr = (sz * (n.value + 1))()
    _check(L.bt_gpt2_param_offsets(_c.byref(c), arr, _c.byref(n)), "bt_gpt2_param_offsets")
    return [int(x) for x in arr]


class GPT2:
    """Device state of one GPT-2 training run: flat params, grads, [m | v]
    and the activation workspace, all torch-allocated; the step runs in
    libbt (bt_gpt2_*)."""

    def __init__(self, cfg, hp, max_B: int, max_T: int, device="cuda", stream=None):
        torch = _torch()
        L = lib()
        self.cfg, self.hp = cfg, hp
        self.max_B, self.max_T = max_B, max_T
        self._ccfg = make_config(cfg, hp)
        self.P = L.bt_gpt2_num_params(_c.byref(self._ccfg))
        if self.P == 0:
            raise ValueError("bad GPT-2 configuration")
        self.n_decay = L.bt_gpt2_num_decay_params(_c.byref(self._ccfg))
        self.params = torch.zeros(self.P, dtype=torch.float32, device=device)
        self.grads = torch.zeros(self.P, dtype=torch.float32, device=device)
        self.opt_state = torch.zeros(2 * self.P, dtype=torch.float32, device=device)
        self.ws_bytes = L.bt_gpt2_workspace_bytes(_c.byref(self._ccfg), max_B, max_T)
        self.workspace = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        base = self.workspace.data_ptr()
        self._ws_ptr = (base + 255) // 256 * 256
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        ctx = vp()
        _check(L.bt_gpt2_create(_c.byref(self._ccfg), self._ws_ptr, self.ws_bytes, max_B, max_T,
                                self.stream.cuda_stream, _c.byref(ctx)), "bt_gpt2_create")
        self._ctx = ctx

    def __del__(self):
        try:
            if getattr(self, "_ctx", None) is not None and _lib is not None:
                _lib.bt_gpt2_destroy(self._ctx)
                self._ctx = None
        except Exception:
            pass

    @property
    def m(self):
        return self.opt_state[: self.P]

    @property
    def v(self):
        return self.opt_state[self.P:]

    def load_params(self, flat: np.ndarray):
        torch = _torch()
        assert flat.dtype == np.float32 and flat.size == self.P
        self.params.copy_(torch.from_numpy(flat))

    @property
    def step_count(self) -> int:
        return lib().bt_gpt2_step_count(self._ctx)

    @step_count.setter
    def step_count(self, t: int):
        lib().bt_gpt2_set_step_count(self._ctx, t)

    def train_step(self, tokens, targets) -> float:
        B, T = tokens.shape
        L = lib()
        loss = L.bt_gpt2_train_step(self._ctx, _p(self.params), _p(self.grads), _p(self.opt_state),
                                    _p(tokens), _p(targets), B, T)
        status = L.bt_last_status()
        if status == BT_ENONFINITE:
            raise BTNonFiniteError(status, "bt_gpt2_train_step", L.bt_last_error().decode())
        if status != 0:
            raise BTError(status, "bt_gpt2_train_step", L.bt_last_error().decode())
        return float(loss)

    def fwd_bwd(self, tokens, targets, loss_scale, accumulate, d_loss, loss_rows=None):
        B, T = tokens.shape
        _check(lib().bt_gpt2_fwd_bwd(self._ctx, _p(self.params), _p(self.grads), _p(tokens), _p(targets),
                                     B, T, loss_scale, int(accumulate), _p(d_loss), _p(loss_rows)),
               "bt_gpt2_fwd_bwd")

    def optimizer_step(self, t: int, lr: float):
        _check(lib().bt_gpt2_optimizer_step(self._ctx, _p(self.params), _p(self.grads), _p(self.opt_state),
                                            t, lr), "bt_gpt2_optimizer_step")

    def read_scalars(self):
        """(last train-step loss, gradient norm, clip coefficient) from the device."""
        out = (f32 * 3)()
        _check(lib().bt_gpt2_read_scalars(self._ctx, out), "bt_gpt2_read_scalars")
        return tuple(float(x) for x in out)

    def profile_enable(self, on: bool = True):
        _check(lib().bt_gpt2_profile_enable(self._ctx, int(on)), "bt_gpt2_profile_enable")

    def profile_read(self, reset: bool = True):
        """Per kernel class: dict(launches, ms, flops, bytes) accumulated since the last reset."""
        arr = (KernelStat * len(PROF_CLASSES))()
        _check(lib().bt_gpt2_profile_read(self._ctx, arr, int(reset)), "bt_gpt2_profile_read")
        return {name: dict(launches=int(s.launches), ms=float(s.ms), flops=float(s.flops), bytes=float(s.bytes))
                for name, s in zip(PROF_CLASSES, arr)}
