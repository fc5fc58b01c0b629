"""Thin torch binding of the BSA C ABI (argument marshalling only).

Torch provides device memory and the current stream; every step of the layer runs in the
HIP kernels of libbsa.so. Function names follow the C entry points of include/bsa.h.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import math

import torch

from . import _lib
from ._lib import BSA_BF16, BSA_F32, BSA_POOL_MEAN, BSA_POOL_MLP, BSA_QC_MEAN, BSA_QC_MLP, check

__all__ = ["Params", "Saved", "build_ball_tree", "build_ball_tree_noalloc", "permute", "unpermute", "sizes", "forward", "backward",
           "block_sizes", "BlockSaved", "block_forward", "block_backward", "BLOCK_WEIGHTS",
           "BSA_F32", "BSA_BF16", "BSA_POOL_MLP", "BSA_POOL_MEAN", "BSA_QC_MEAN", "BSA_QC_MLP"]


@dataclasses.dataclass
class Params:
    batch: int
    n: int
    heads: int
    head_dim: int
    ball_size: int
    cmp_block: int
    slc_block: int
    topk: int
    group_size: int
    cmp_stride: int | None = None
    mask_own_ball: int = 1
    store_lse: int = 1
    deterministic: int = 1
    kv_pool: int = BSA_POOL_MLP
    dtype: int = BSA_BF16
    softmax_scale: float = 0.0
    q_coarsen: int = BSA_QC_MEAN
    group_compression: int = 0

    def c(self) -> _lib.bsa_params_t:
        return _lib.bsa_params_t(
            self.batch, self.n, self.heads, self.head_dim, self.ball_size, self.cmp_block,
            self.cmp_block if self.cmp_stride is None else self.cmp_stride, self.slc_block, self.topk,
            self.group_size, self.mask_own_ball, self.store_lse, self.deterministic, self.kv_pool,
            self.dtype, self.softmax_scale, self.q_coarsen, self.group_compression)

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.bfloat16 if self.dtype == BSA_BF16 else torch.float32

    @classmethod
    def from_config(cls, cfg, **kw) -> "Params":
        return cls(batch=cfg.batch, n=cfg.n_pad, heads=cfg.heads, head_dim=cfg.head_dim, ball_size=cfg.ball,
                   cmp_block=cfg.cmp_block, cmp_stride=cfg.cmp_stride, slc_block=cfg.slc_block, topk=cfg.topk,
                   group_size=cfg.group, dtype=BSA_BF16 if cfg.dtype == "bf16" else BSA_F32, **kw)


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def _require(t, name, dtype, shape=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def build_ball_tree(points: torch.Tensor, n_pad: int, stream=None) -> torch.Tensor:
    """Slot -> point permutation [B, n_pad] int32 (-1 = padding) of clouds [B, n_real, dim] f32."""
    lib = _lib.load()
    _require(points, "points", torch.float32)
    B, n_real, dim = points.shape
    ws_bytes = lib.bsa_ball_tree_workspace_bytes(n_real, n_pad, dim, B)
    if ws_bytes == 0:
        raise ValueError("invalid ball-tree sizes")
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=points.device)
    perm = torch.empty((B, n_pad), dtype=torch.int32, device=points.device)
    check(lib.bsa_build_ball_tree(_ptr(points), n_real, dim, n_pad, B, _ptr(perm), _ptr(ws), ws_bytes,
                                  _stream(stream)), "bsa_build_ball_tree")
    return perm


def build_ball_tree_noalloc(points: torch.Tensor, perm: torch.Tensor, stream=None) -> torch.Tensor:
    """bsa_build_ball_tree_noalloc: fills the caller's perm [B, n_pad] int32 from clouds
    [B, n_real, dim] f32 using the library's static scratch (no workspace, no allocation)."""
    lib = _lib.load()
    _require(points, "points", torch.float32)
    _require(perm, "perm", torch.int32)
    B, n_real, dim = points.shape
    if perm.dim() != 2 or perm.shape[0] != B:
        raise ValueError("perm must be [B, n_pad]")
    check(lib.bsa_build_ball_tree_noalloc(_ptr(points), n_real, dim, perm.shape[1], B, _ptr(perm), _stream(stream)),
          "bsa_build_ball_tree_noalloc")
    return perm


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return BSA_F32
    if t.dtype == torch.bfloat16:
        return BSA_BF16
    raise ValueError("only float32 and bfloat16 are supported")


def permute(src: torch.Tensor, perm: torch.Tensor, heads: int, head_dim: int, with_valid: bool = False,
            stream=None):
    """[B, n_real, heads*head_dim] -> [B, heads, n_pad, head_dim] in ball order (+ valid [B, n_pad] u8)."""
    lib = _lib.load()
    B, n_real, cols = src.shape
    assert cols == heads * head_dim
    _require(src, "src", src.dtype)
    _require(perm, "perm", torch.int32)
    n_pad = perm.shape[1]
    dst = torch.empty((B, heads, n_pad, head_dim), dtype=src.dtype, device=src.device)
    valid = torch.empty((B, n_pad), dtype=torch.uint8, device=src.device) if with_valid else None
    check(lib.bsa_permute(_ptr(src), _ptr(perm), n_real, n_pad, B, heads, head_dim, _dtype_code(src), _ptr(dst),
                          _ptr(valid), _stream(stream)), "bsa_permute")
    return (dst, valid) if with_valid else dst


def unpermute(src: torch.Tensor, perm: torch.Tensor, n_real: int, stream=None) -> torch.Tensor:
    """[B, heads, n_pad, head_dim] in ball order -> [B, n_real, heads*head_dim]."""
    lib = _lib.load()
    B, heads, n_pad, hd = src.shape
    _require(src, "src", src.dtype)
    _require(perm, "perm", torch.int32)
    dst = torch.empty((B, n_real, heads * hd), dtype=src.dtype, device=src.device)
    check(lib.bsa_unpermute(_ptr(src), _ptr(perm), n_real, n_pad, B, heads, hd, _dtype_code(src), _ptr(dst),
                            _stream(stream)), "bsa_unpermute")
    return dst


def sizes(p: Params):
    """(forward workspace, backward workspace, saved) byte counts; raises on invalid params."""
    lib = _lib.load()
    a, b, c = C.c_size_t(), C.c_size_t(), C.c_size_t()
    cp = p.c()
    check(lib.bsa_sizes(C.byref(cp), C.byref(a), C.byref(b), C.byref(c)), "bsa_sizes")
    return a.value, b.value, c.value


class Saved:
    """Tensors saved by forward(): one device buffer plus typed views of its parts."""

    def __init__(self, p: Params, device):
        lib = _lib.load()
        _, _, nbytes = sizes(p)
        self.p = p
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.c = _lib.bsa_saved_t()
        cp = p.c()
        check(lib.bsa_saved_view(C.byref(cp), _ptr(self.buf), C.byref(self.c)), "bsa_saved_view")
        base = self.buf.data_ptr()
        B, H, N, d = p.batch, p.heads, p.n, p.head_dim

        def view(ptr, dtype, shape):
            off = ptr - base
            count = math.prod(shape)
            esz = torch.empty((), dtype=dtype).element_size()
            return self.buf[off:off + count * esz].view(dtype).view(shape)

        self.sel_idx = view(self.c.sel_idx, torch.int32, (B, H, N // p.group_size, p.topk))
        # store_lse = 0: the statistics are not kept (the backward recomputes them)
        self.lse = view(self.c.lse, torch.float32, (3, B, H, N)) if self.c.lse else None
        self.o_branch = view(self.c.o_branch, p.torch_dtype, (2, B, H, N, d))   # ball, selection
        self.o_cmp = view(self.c.o_cmp, torch.float32, (B, H, N, d))
        self.kcmp = view(self.c.kcmp, torch.float32, (B, H, N // p.cmp_block, d))
        self.vcmp = view(self.c.vcmp, torch.float32, (B, H, N // p.cmp_block, d))
        self.hid_k = view(self.c.hid_k, torch.float32, (B, H, N // p.cmp_block, d))
        self.hid_v = view(self.c.hid_v, torch.float32, (B, H, N // p.cmp_block, d))
        self.cvalid = view(self.c.cvalid, torch.uint8, (B, N // p.cmp_block))
        self.qcmp = view(self.c.qcmp, torch.float32, (B, H, N // p.group_size, d))
        self.hid_q = view(self.c.hid_q, torch.float32, (B, H, N // p.cmp_block, d)) if self.c.hid_q else None
        self.ocmp = view(self.c.ocmp, torch.float32, (B, H, N // p.cmp_block, d)) if self.c.ocmp else None


    def branch_outputs(self) -> torch.Tensor:
        """The three branch outputs as one float32 [3, B, H, N, d] tensor (ball, compression,
        selection); a copy, for inspection."""
        return torch.stack([self.o_branch[0].float(), self.o_cmp, self.o_branch[1].float()])


def _mlp(phi):
    if phi is None:
        return None
    for w in ("w1", "b1", "w2", "b2"):
        _require(phi[w], f"phi.{w}", torch.float32)
    return _lib.bsa_mlp_t(phi["w1"].data_ptr(), phi["b1"].data_ptr(), phi["w2"].data_ptr(), phi["b2"].data_ptr())


def forward(p: Params, q, k, v, valid, gate, phi_k, phi_v, saved: Saved | None = None, stream=None, phi_q=None):
    """Layer forward. Returns (o, saved). phi_q: the query-coarsening MLP (BSA_QC_MLP)."""
    lib = _lib.load()
    shape = (p.batch, p.heads, p.n, p.head_dim)
    for name, t in (("q", q), ("k", k), ("v", v)):
        _require(t, name, p.torch_dtype, shape)
    _require(gate, "gate", torch.float32, (p.batch, p.n, 3))
    if valid is not None:
        _require(valid, "valid", torch.uint8, (p.batch, p.n))
    ws_bytes, _, _ = sizes(p)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=q.device)
    saved = saved or Saved(p, q.device)
    o = torch.empty(shape, dtype=p.torch_dtype, device=q.device)
    mk, mv, mq = _mlp(phi_k), _mlp(phi_v), _mlp(phi_q)
    cp = p.c()
    check(lib.bsa_forward(C.byref(cp), _ptr(q), _ptr(k), _ptr(v), _ptr(valid), _ptr(gate),
                          C.byref(mk) if mk else None, C.byref(mv) if mv else None, C.byref(mq) if mq else None,
                          _ptr(o), C.byref(saved.c), _ptr(ws), ws_bytes, _stream(stream)), "bsa_forward")
    return o, saved


def backward(p: Params, q, k, v, valid, gate, phi_k, phi_v, saved: Saved, d_o, stream=None, phi_q=None):
    """Layer backward. Returns dict(dq, dk, dv, dgate, dphi_k, dphi_v, dphi_q) (float32); dphi_q is
    filled only with group compression and MLP query coarsening."""
    lib = _lib.load()
    shape = (p.batch, p.heads, p.n, p.head_dim)
    for name, t in (("q", q), ("k", k), ("v", v), ("d_o", d_o)):
        _require(t, name, p.torch_dtype, shape)
    _require(gate, "gate", torch.float32, (p.batch, p.n, 3))
    dev = q.device
    _, ws_bytes, _ = sizes(p)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    dq = torch.empty(shape, dtype=torch.float32, device=dev)
    dk = torch.empty_like(dq)
    dv = torch.empty_like(dq)
    dgate = torch.empty((p.batch, p.n, 3), dtype=torch.float32, device=dev)
    grads = {}
    cgr = []
    q_grad = p.group_compression and p.q_coarsen == BSA_QC_MLP
    for name, phi, on in (("dphi_k", phi_k, p.kv_pool == BSA_POOL_MLP), ("dphi_v", phi_v, p.kv_pool == BSA_POOL_MLP),
                          ("dphi_q", phi_q, q_grad)):
        if on:
            g = {w: torch.empty_like(phi[w]) for w in ("w1", "b1", "w2", "b2")}
            grads[name] = g
            cgr.append(_lib.bsa_mlp_t(g["w1"].data_ptr(), g["b1"].data_ptr(), g["w2"].data_ptr(), g["b2"].data_ptr()))
        else:
            grads[name] = {}
            cgr.append(None)
    mk, mv, mq = _mlp(phi_k), _mlp(phi_v), _mlp(phi_q)
    cp = p.c()
    check(lib.bsa_backward(C.byref(cp), _ptr(q), _ptr(k), _ptr(v), _ptr(valid), _ptr(gate),
                           C.byref(mk) if mk else None, C.byref(mv) if mv else None, C.byref(mq) if mq else None,
                           C.byref(saved.c), _ptr(d_o), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dgate),
                           C.byref(cgr[0]) if cgr[0] else None, C.byref(cgr[1]) if cgr[1] else None,
                           C.byref(cgr[2]) if cgr[2] else None, _ptr(ws), ws_bytes, _stream(stream)),
          "bsa_backward")
    grads.update(dq=dq, dk=dk, dv=dv, dgate=dgate)
    return grads


# ---- the transformer block around the layer (bsa_block_* in include/bsa.h) ----

BLOCK_WEIGHTS = _lib._BLOCK_W


def block_sizes(p: Params, ffn: int):
    """(forward workspace, backward workspace, saved) byte counts of one block."""
    lib = _lib.load()
    a, b, c = C.c_size_t(), C.c_size_t(), C.c_size_t()
    cp = p.c()
    check(lib.bsa_block_sizes(C.byref(cp), ffn, C.byref(a), C.byref(b), C.byref(c)), "bsa_block_sizes")
    return a.value, b.value, c.value


class BlockSaved:
    """Tensors saved by block_forward(): one device buffer plus typed views of its parts."""

    def __init__(self, p: Params, ffn: int, device):
        lib = _lib.load()
        _, _, nbytes = block_sizes(p, ffn)
        self.p, self.ffn = p, ffn
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.c = _lib.bsa_block_saved_t()
        cp = p.c()
        check(lib.bsa_block_saved_view(C.byref(cp), ffn, _ptr(self.buf), C.byref(self.c)), "bsa_block_saved_view")
        base = self.buf.data_ptr()
        B, H, N, d = p.batch, p.heads, p.n, p.head_dim
        Cc = H * d

        def view(ptr, dtype, shape):
            off = ptr - base
            esz = torch.empty((), dtype=dtype).element_size()
            return self.buf[off:off + math.prod(shape) * esz].view(dtype).view(shape)

        bf, f32 = torch.bfloat16, torch.float32
        self.rstd1 = view(self.c.rstd1, f32, (B, N))
        self.rstd2 = view(self.c.rstd2, f32, (B, N))
        self.xn1 = view(self.c.xn1, bf, (B, N, Cc))
        self.gate = view(self.c.gate, f32, (B, N, 3))
        self.q, self.k, self.v, self.o = (view(getattr(self.c, n), bf, (B, H, N, d)) for n in ("q", "k", "v", "o"))
        self.h = view(self.c.h, f32, (B, N, Cc))
        self.xn2 = view(self.c.xn2, bf, (B, N, Cc))
        self.uw = view(self.c.uw, bf, (B, N, 2 * ffn))
        self.a = view(self.c.a, bf, (B, N, ffn))
        self.sel_idx = view(self.c.layer.sel_idx, torch.int32, (B, H, N // p.group_size, p.topk))


def _mlp_struct(phi):
    return _mlp(phi) if phi else _lib.bsa_mlp_t()


def _block_weights(p: Params, ffn: int, W, phi_k, phi_v, phi_q):
    Cc = p.heads * p.head_dim
    shapes = {"g1": (Cc,), "wqkv": (3 * Cc, Cc), "wg": (3, Cc), "wo": (Cc, Cc), "g2": (Cc,), "w1": (ffn, Cc),
              "w3": (ffn, Cc), "w2": (Cc, ffn)}
    for n in BLOCK_WEIGHTS:
        _require(W[n], n, torch.float32, shapes[n])
    return _lib.bsa_block_weights_t(*[W[n].data_ptr() for n in BLOCK_WEIGHTS], _mlp_struct(phi_k), _mlp_struct(phi_v),
                                    _mlp_struct(phi_q))


def block_forward(p: Params, ffn: int, W, phi_k, phi_v, x, valid=None, saved: BlockSaved | None = None, phi_q=None,
                  stream=None):
    """One block forward: x [B, N, C] float32 -> (y, saved). W: dict of float32 weights
    (BLOCK_WEIGHTS); phi_*: the layer's MLPs."""
    lib = _lib.load()
    Cc = p.heads * p.head_dim
    _require(x, "x", torch.float32, (p.batch, p.n, Cc))
    if valid is not None:
        _require(valid, "valid", torch.uint8, (p.batch, p.n))
    cw = _block_weights(p, ffn, W, phi_k, phi_v, phi_q)
    ws_bytes, _, _ = block_sizes(p, ffn)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=x.device)
    saved = saved or BlockSaved(p, ffn, x.device)
    y = torch.empty_like(x)
    cp = p.c()
    check(lib.bsa_block_forward(C.byref(cp), ffn, C.byref(cw), _ptr(x), _ptr(valid), _ptr(y), C.byref(saved.c),
                                _ptr(ws), ws_bytes, _stream(stream)), "bsa_block_forward")
    return y, saved


def block_backward(p: Params, ffn: int, W, phi_k, phi_v, x, saved: BlockSaved, dy, valid=None, phi_q=None,
                   stream=None):
    """One block backward: returns dict(dx, dW: {name: grad}, dphi_k, dphi_v, dphi_q) (float32)."""
    lib = _lib.load()
    Cc = p.heads * p.head_dim
    _require(x, "x", torch.float32, (p.batch, p.n, Cc))
    _require(dy, "dy", torch.float32, (p.batch, p.n, Cc))
    cw = _block_weights(p, ffn, W, phi_k, phi_v, phi_q)
    dev = x.device
    _, ws_bytes, _ = block_sizes(p, ffn)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    dW = {n: torch.empty_like(W[n]) for n in BLOCK_WEIGHTS}
    grads = {}
    structs = []
    q_grad = p.group_compression and p.q_coarsen == BSA_QC_MLP
    for name, phi, on in (("dphi_k", phi_k, p.kv_pool == BSA_POOL_MLP), ("dphi_v", phi_v, p.kv_pool == BSA_POOL_MLP),
                          ("dphi_q", phi_q, q_grad)):
        g = {w: torch.empty_like(phi[w]) for w in ("w1", "b1", "w2", "b2")} if on else {}
        grads[name] = g
        structs.append(_mlp_struct(g))
    cg = _lib.bsa_block_grads_t(*[dW[n].data_ptr() for n in BLOCK_WEIGHTS], *structs)
    dx = torch.empty_like(x)
    cp = p.c()
    check(lib.bsa_block_backward(C.byref(cp), ffn, C.byref(cw), _ptr(x), _ptr(valid), C.byref(saved.c), _ptr(dy),
                                 _ptr(dx), C.byref(cg), _ptr(ws), ws_bytes, _stream(stream)), "bsa_block_backward")
    grads.update(dx=dx, dW=dW)
    return grads
