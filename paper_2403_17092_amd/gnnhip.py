"""Python binding of libgnnhip.so (ctypes).

Argument marshalling only: every step of the training path runs in the HIP
kernels of the library.  PyTorch supplies device memory (tensors) and the
stream (torch.cuda.current_stream()).  The names follow the C ABI in
include/gnnhip.h without the ``gnn_`` prefix.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgnnhip.so")

OK, EINVAL, EWORKSPACE, EHIP, EDEVICE = 0, -1, -2, -3, -4
F32, BF16 = 0, 1
SAGE_MEAN, GCN, GIN, GAT = 0, 1, 2, 3
DEVERR_SEED_RANGE, DEVERR_LABEL_RANGE, DEVERR_CAPACITY, DEVERR_GRAPH, DEVERR_SYNC = 1, 2, 4, 8, 16
MAX_LAYERS = 4
STAGES = ["sample", "gather", "agg1", "gemm1", "fwd_rest", "backward", "sgd"]

KIND = {"sage_mean": SAGE_MEAN, "gcn": GCN, "gin": GIN, "gat": GAT}


class GnnError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"gnnhip error {code}: {msg}")
        self.code = code


class CCsr(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int64), ("num_edges", ctypes.c_int64),
                ("rowptr", ctypes.c_void_p), ("rowptr_bits", ctypes.c_int32),
                ("col", ctypes.c_void_p), ("scan_order", ctypes.c_int32),
                ("hub_degree", ctypes.c_int32)]


class CBlock(ctypes.Structure):
    _fields_ = [("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p),
                ("src_nodes", ctypes.c_void_p), ("src_occ", ctypes.c_void_p),
                ("counts", ctypes.c_void_p), ("cap_dst", ctypes.c_int32),
                ("cap_src", ctypes.c_int32), ("cap_edges", ctypes.c_int64)]


OPT_SGD, OPT_ADAM = 0, 1


class COptimizer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("m", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("steps", ctypes.c_int64)]


class CModel(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("num_layers", ctypes.c_int32),
                ("dims", ctypes.c_int32 * (MAX_LAYERS + 1)), ("weights", ctypes.c_void_p),
                ("opt", ctypes.POINTER(COptimizer))]


class CTrainViews(ctypes.Structure):
    _fields_ = [("blocks", CBlock * MAX_LAYERS), ("xg", ctypes.c_void_p),
                ("x", ctypes.c_void_p * MAX_LAYERS), ("x_ld", ctypes.c_int32 * MAX_LAYERS),
                ("x_dtype", ctypes.c_int32 * MAX_LAYERS), ("h", ctypes.c_void_p * MAX_LAYERS),
                ("dweights", ctypes.c_void_p), ("dlogits", ctypes.c_void_p),
                ("comp_ptr", ctypes.c_void_p)]


class CFeatureCache(ctypes.Structure):
    _fields_ = [("num_sets", ctypes.c_int32), ("ways", ctypes.c_int32), ("width", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("mem", ctypes.c_void_p)]


class CTrace(ctypes.Structure):
    _fields_ = [("events", ctypes.c_void_p), ("names", ctypes.c_void_p), ("only", ctypes.c_char_p),
                ("capacity", ctypes.c_int32), ("count", ctypes.c_int32),
                ("dropped", ctypes.c_int32)]


_lib = None


def lib():
    """The loaded library.  Raises if it has not been built: there is no fallback."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing; build it with "
                          "`python -m paper_2403_17092_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, u64, sz, f32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                 ctypes.c_uint64, ctypes.c_size_t, ctypes.c_float)
    pi32 = ctypes.POINTER(ctypes.c_int32)
    pi64 = ctypes.POINTER(ctypes.c_int64)
    sig = {
        "gnn_num_params": (i64, [ctypes.POINTER(CModel)]),
        "gnn_block_caps": (ctypes.c_int, [i32, pi32, i32, i64, pi32, pi32, pi64]),
        "gnn_sample_workspace_bytes": (sz, [i32, pi32, i32, i64]),
        "gnn_sample_blocks": (ctypes.c_int, [ctypes.POINTER(CCsr), P, i32, pi32, i32, u64,
                                             ctypes.POINTER(CBlock), P, sz, P]),
        "gnn_gather_features": (ctypes.c_int, [P, i32, i64, i64, i32, P, P, i32, P, i64, P]),
        "gnn_layer_fwd": (ctypes.c_int, [ctypes.POINTER(CBlock), i32, P, i32, i32, P, i32, i32, P,
                                         P, P]),
        "gnn_layer_bwd_workspace_bytes": (sz, [i32, i32]),
        "gnn_layer_bwd": (ctypes.c_int, [ctypes.POINTER(CBlock), i32, i32, P, P, P, i32, P, P, P,
                                         i32, P, sz, P]),
        "gnn_loss_workspace_bytes": (sz, [i32]),
        "gnn_softmax_xent": (ctypes.c_int, [P, P, i32, i32, P, P, P, sz, P]),
        "gnn_softmax_xent_noalloc": (ctypes.c_int, [P, P, i32, i32, P, P, P]),
        "gnn_sgd": (ctypes.c_int, [P, P, i64, f32, P]),
        "gnn_train_workspace_bytes": (sz, [ctypes.POINTER(CModel), i32, i32, pi32, i64]),
        "gnn_train_step": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P, i32, i64,
                                          P, P, i32, pi32, u64, f32, P, P, sz, P]),
        "gnn_train_step_ex": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P, i32,
                                             i64, P, P, i32, pi32, u64, f32, P, P, sz, P, P]),
        "gnn_train_step_views": (ctypes.c_int, [ctypes.POINTER(CModel), i32, i32, pi32, i64, P, sz,
                                                ctypes.POINTER(CTrainViews)]),
        "gnn_train_slot_views": (ctypes.c_int, [ctypes.POINTER(CModel), i32, i32, pi32, i64, P, sz,
                                                i32, ctypes.POINTER(CTrainViews)]),
        "gnn_shadow_caps": (ctypes.c_int, [i32, i32, i32, pi32, pi64]),
        "gnn_shadow_workspace_bytes": (sz, [i32, i32, i32]),
        "gnn_sample_shadow": (ctypes.c_int, [ctypes.POINTER(CCsr), P, i32, i32, i32, u64,
                                             ctypes.POINTER(CBlock), P, P, P, sz, P]),
        "gnn_shadow_train_workspace_bytes": (sz, [ctypes.POINTER(CModel), i32, i32, i32, i32]),
        "gnn_shadow_train_step": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P,
                                                 i32, i64, P, P, i32, i32, i32, u64, f32, P, P, sz,
                                                 P, P]),
        "gnn_shadow_train_step_views": (ctypes.c_int, [ctypes.POINTER(CModel), i32, i32, i32, i32,
                                                       P, sz, ctypes.POINTER(CTrainViews)]),
        "gnn_train_sample": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P, i32, i64,
                                            P, i32, pi32, u64, P, sz, i32, P]),
        "gnn_train_model": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P, i32, i64,
                                           P, P, i32, pi32, f32, P, P, sz, i32, P, P]),
        "gnn_shadow_train_sample": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P,
                                                   i32, i64, P, i32, i32, i32, u64, P, sz, i32, P]),
        "gnn_shadow_train_model": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P,
                                                  i32, i64, P, P, i32, i32, i32, f32, P, P, sz, i32,
                                                  P, P]),
        "gnn_train_pipelined": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P, i32,
                                               i64, P, P, P, i32, i32, pi32, f32, P, P, sz, P, P, P]),
        "gnn_shadow_train_pipelined": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr),
                                                      P, i32, i64, P, P, P, i32, i32, i32, i32, f32,
                                                      P, P, sz, P, P, P]),
        "gnn_check_errors": (ctypes.c_int, [P, pi32]),
        "gnn_last_error": (ctypes.c_char_p, []),
        "gnn_version": (ctypes.c_char_p, []),
        "gnn_trace_begin": (ctypes.c_int, [ctypes.POINTER(CTrace)]),
        "gnn_estimate_workspace_bytes": (sz, [i32, pi32, i32, i64]),
        "gnn_estimate_work": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P, P, i32,
                                             i32, pi32, P, P, P, sz, P]),
        "gnn_shadow_estimate_workspace_bytes": (sz, [i32, i32, i32]),
        "gnn_shadow_estimate_work": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P,
                                                    P, i32, i32, i32, i32, P, P, P, sz, P]),
        "gnn_dlb_assign": (ctypes.c_int, [pi64, i32, ctypes.POINTER(ctypes.c_double), i32, pi32,
                                          pi64]),
        "gnn_feature_cache_bytes": (sz, [i32, i32, i32, i32]),
        "gnn_feature_cache_reset": (ctypes.c_int, [ctypes.POINTER(CFeatureCache), P]),
        "gnn_feature_cache_views": (ctypes.c_int, [ctypes.POINTER(CFeatureCache),
                                                   ctypes.POINTER(ctypes.c_void_p),
                                                   ctypes.POINTER(ctypes.c_void_p),
                                                   ctypes.POINTER(ctypes.c_void_p)]),
        "gnn_gather_cached_workspace_bytes": (sz, [i32, i32]),
        "gnn_train_cached_workspace_bytes": (sz, [ctypes.POINTER(CModel), i32, i32, pi32, i64, i32]),
        "gnn_train_step_cached": (ctypes.c_int, [ctypes.POINTER(CModel), ctypes.POINTER(CCsr), P, i32,
                                                 i64, ctypes.POINTER(CFeatureCache), P, P, P, i32,
                                                 pi32, u64, f32, P, P, sz, P]),
        "gnn_gather_cached": (ctypes.c_int, [ctypes.POINTER(CFeatureCache), P, i64, i64, P, P, i32,
                                             P, i64, P, P, sz, P]),
        "gnn_dlb_ratio": (ctypes.c_int, [pi64, ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_double), i32, ctypes.c_double,
                                         ctypes.POINTER(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


class _HipEvents:
    """HIP events (timing disabled) created through the HIP runtime torch uses."""

    def __init__(self, n: int):
        self._rt = ctypes.CDLL("libamdhip64.so", mode=ctypes.RTLD_GLOBAL)
        self._rt.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self._rt.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.array = (ctypes.c_void_p * n)()
        for i in range(n):
            e = ctypes.c_void_p()
            if self._rt.hipEventCreateWithFlags(ctypes.byref(e), 2) != 0:  # hipEventDisableTiming
                raise GnnError(EHIP, "hipEventCreateWithFlags failed")
            self.array[i] = e.value

    def __del__(self):
        try:
            for e in self.array:
                if e:
                    self._rt.hipEventDestroy(ctypes.c_void_p(e))
        except Exception:
            pass


def _check(rc: int):
    if rc != OK:
        raise GnnError(rc, lib().gnn_last_error().decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _i32arr(xs: Sequence[int]):
    return (ctypes.c_int32 * len(xs))(*[int(x) for x in xs])


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return BF16
    raise TypeError(f"unsupported feature dtype {t.dtype}")


# ---------------------------------------------------------------------------
# graph and blocks
# ---------------------------------------------------------------------------
@dataclass
class Csr:
    rowptr: torch.Tensor  # int32 or int64, [N + 1]
    col: torch.Tensor     # int32, [E]
    # schedule options (gnn_csr): 1 takes every sampler scan tile by ticket;
    # ShaDow's row-search degree (0: the default)
    scan_order: int = 0
    hub_degree: int = 0
    c: CCsr = field(init=False)

    def __post_init__(self):
        assert self.col.dtype == torch.int32
        bits = 64 if self.rowptr.dtype == torch.int64 else 32
        self.c = CCsr(self.rowptr.shape[0] - 1, self.col.shape[0], self.rowptr.data_ptr(), bits,
                      self.col.data_ptr(), self.scan_order, self.hub_degree)

    @property
    def num_nodes(self) -> int:
        return int(self.rowptr.shape[0] - 1)


def block_caps(B: int, fanouts: Sequence[int], N: int):
    L = len(fanouts)
    cd, cs = (ctypes.c_int32 * L)(), (ctypes.c_int32 * L)()
    ce = (ctypes.c_int64 * L)()
    _check(lib().gnn_block_caps(B, _i32arr(fanouts), L, N, cd, cs, ce))
    return list(cd), list(cs), list(ce)


@dataclass
class Block:
    indptr: torch.Tensor
    indices: torch.Tensor
    src_nodes: torch.Tensor
    src_occ: torch.Tensor
    counts: torch.Tensor
    cap_dst: int
    cap_src: int
    cap_edges: int

    def cstruct(self) -> CBlock:
        return CBlock(self.indptr.data_ptr(), self.indices.data_ptr(), self.src_nodes.data_ptr(),
                      self.src_occ.data_ptr(), self.counts.data_ptr(), self.cap_dst, self.cap_src,
                      self.cap_edges)

    @staticmethod
    def from_ws(cb: CBlock, ws: torch.Tensor) -> "Block":
        """A Block whose tensors alias the workspace memory described by a C struct."""
        def view(ptr, n):
            return ws_view(ws, ptr, n, torch.int32)
        return Block(view(cb.indptr, cb.cap_dst + 1), view(cb.indices, max(1, cb.cap_edges)),
                     view(cb.src_nodes, max(1, cb.cap_src)), view(cb.src_occ, max(1, cb.cap_src)),
                     view(cb.counts, 4), cb.cap_dst, cb.cap_src, cb.cap_edges)

    def host(self):
        """(n_dst, n_src, n_edges, indptr, indices, src_nodes, src_occ) as numpy, trimmed."""
        c = self.counts.cpu().numpy()
        nd, ns, ne = int(c[0]), int(c[1]), int(c[2])
        return (nd, ns, ne, self.indptr[: nd + 1].cpu().numpy(), self.indices[:ne].cpu().numpy(),
                self.src_nodes[:ns].cpu().numpy(), self.src_occ[:ns].cpu().numpy())


def ws_view(ws: torch.Tensor, ptr: int, n: int, dtype) -> torch.Tensor:
    """n elements of `dtype` at device address ptr inside the uint8 workspace tensor ws."""
    esize = torch.tensor([], dtype=dtype).element_size()
    off = int(ptr) - ws.data_ptr()
    assert 0 <= off and off + n * esize <= ws.numel() and off % esize == 0
    return ws[off: off + n * esize].view(dtype)


def alloc_blocks(B: int, fanouts: Sequence[int], N: int, device="cuda") -> List[Block]:
    cd, cs, ce = block_caps(B, fanouts, N)
    out = []
    for h in range(len(fanouts)):
        kw = dict(dtype=torch.int32, device=device)
        out.append(Block(torch.zeros(cd[h] + 1, **kw), torch.zeros(max(1, ce[h]), **kw),
                         torch.zeros(max(1, cs[h]), **kw), torch.zeros(max(1, cs[h]), **kw),
                         torch.zeros(4, **kw), cd[h], cs[h], ce[h]))
    return out


def sample_workspace_bytes(B: int, fanouts: Sequence[int], N: int) -> int:
    return int(lib().gnn_sample_workspace_bytes(B, _i32arr(fanouts), len(fanouts), N))


def sample_blocks(csr: Csr, seeds: torch.Tensor, fanouts: Sequence[int], rng_key: int,
                  blocks: Optional[List[Block]] = None, ws: Optional[torch.Tensor] = None,
                  stream=None) -> List[Block]:
    """gnn_sample_blocks.  A caller-provided `ws` (uint8, at least
    sample_workspace_bytes) keeps per-node state between calls: reuse it only
    for sampling."""
    B = int(seeds.shape[0])
    assert seeds.dtype == torch.int32 and seeds.is_contiguous()
    if blocks is None:
        blocks = alloc_blocks(B, fanouts, csr.num_nodes, seeds.device)
    if ws is None:
        ws = torch.zeros(sample_workspace_bytes(B, fanouts, csr.num_nodes), dtype=torch.uint8,
                         device=seeds.device)
    cb = (CBlock * len(blocks))(*[b.cstruct() for b in blocks])
    _check(lib().gnn_sample_blocks(ctypes.byref(csr.c), _ptr(seeds), B, _i32arr(fanouts),
                                   len(fanouts), rng_key, cb, _ptr(ws), ws.numel(), _stream(stream)))
    return blocks


def gather_features(X: torch.Tensor, ids: torch.Tensor, n_ids: torch.Tensor, cap: int,
                    out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    F = int(X.shape[1])
    if out is None:
        out = torch.empty((max(1, cap), F), dtype=X.dtype, device=X.device)
    _check(lib().gnn_gather_features(_ptr(X), _dtype_code(X), X.shape[0], X.stride(0), F, _ptr(ids),
                                     _ptr(n_ids), cap, _ptr(out), out.stride(0), _stream(stream)))
    return out


def x_width(kind: int, F_in: int, F_out: int) -> int:
    """Row stride of a layer's GEMM input: [H_dst | agg] for GraphSAGE, agg for
    GCN, [agg | M | pad] for GIN (M = the MLP's hidden rows, padded to a
    multiple of 4 columns)."""
    if kind == GIN:
        return F_in + (F_out + 3) // 4 * 4
    return 2 * F_in if kind == SAGE_MEAN else F_in


def w_rows(kind: int, F_in: int, F_out: int) -> int:
    """Rows of a layer's stacked weights: [W_self; W_neigh], W, [W_a; W_b] or
    [W; a_l; a_r] (GAT)."""
    if kind == GAT:
        return F_in + 2
    return 2 * F_in if kind == SAGE_MEAN else (F_in + F_out if kind == GIN else F_in)


def layer_fwd(blk: Block, kind: int, H_in: torch.Tensor, W: torch.Tensor, relu: bool,
              X_out: Optional[torch.Tensor] = None, H_out: Optional[torch.Tensor] = None,
              stream=None):
    """W: [K_w x F_out], the stacked [W_self; W_neigh] for GraphSAGE, [W_a; W_b]
    for GIN.  Returns (X, H_out)."""
    F_in, F_out = int(H_in.shape[1]), int(W.shape[1])
    dev = H_in.device
    if X_out is None:
        X_out = torch.zeros((max(1, blk.cap_dst), x_width(kind, F_in, F_out)), dtype=torch.float32,
                            device=dev)
    if H_out is None:
        H_out = torch.zeros((max(1, blk.cap_dst), F_out), dtype=torch.float32, device=dev)
    cb = blk.cstruct()
    _check(lib().gnn_layer_fwd(ctypes.byref(cb), kind, _ptr(H_in), _dtype_code(H_in), F_in,
                               _ptr(W), F_out, int(relu), _ptr(X_out), _ptr(H_out), _stream(stream)))
    return X_out, H_out


def layer_bwd(blk: Block, kind: int, F_in: int, X: torch.Tensor, H_in: Optional[torch.Tensor],
              W: torch.Tensor, dZ: torch.Tensor, want_dH: bool, mask_relu: bool, stream=None):
    """Returns (dW [K_w x F_out], dH_in or None)."""
    F_out = int(W.shape[1])
    dev = X.device
    dW = torch.empty((w_rows(kind, F_in, F_out), F_out), dtype=torch.float32, device=dev)
    dH = torch.empty((max(1, blk.cap_src), F_in), dtype=torch.float32, device=dev) if want_dH else None
    ws_cols = 2 * F_in + F_out + 4 if kind == GIN else F_in
    wsb = int(lib().gnn_layer_bwd_workspace_bytes(blk.cap_dst, ws_cols))
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    cb = blk.cstruct()
    _check(lib().gnn_layer_bwd(ctypes.byref(cb), kind, F_in, _ptr(X), _ptr(H_in), _ptr(W), F_out,
                               _ptr(dZ), _ptr(dW), _ptr(dH), int(mask_relu), _ptr(ws), wsb,
                               _stream(stream)))
    return dW, dH


def softmax_xent(logits: torch.Tensor, labels: torch.Tensor, stream=None):
    B, C = int(logits.shape[0]), int(logits.shape[1])
    dl = torch.empty_like(logits)
    loss = torch.zeros(1, dtype=torch.float32, device=logits.device)
    wsb = int(lib().gnn_loss_workspace_bytes(B))
    ws = torch.empty(wsb, dtype=torch.uint8, device=logits.device)
    _check(lib().gnn_softmax_xent(_ptr(logits), _ptr(labels), B, C, _ptr(dl), _ptr(loss), _ptr(ws),
                                  wsb, _stream(stream)))
    return loss, dl


def softmax_xent_noalloc(logits: torch.Tensor, labels: torch.Tensor, dlogits: torch.Tensor,
                         loss: torch.Tensor, stream=None):
    """gnn_softmax_xent_noalloc into caller-made dlogits [B x C] and loss [1]."""
    B, C = int(logits.shape[0]), int(logits.shape[1])
    _check(lib().gnn_softmax_xent_noalloc(_ptr(logits), _ptr(labels), B, C, _ptr(dlogits), _ptr(loss),
                                          _stream(stream)))
    return loss, dlogits


def sgd(w: torch.Tensor, g: torch.Tensor, lr: float, stream=None):
    _check(lib().gnn_sgd(_ptr(w), _ptr(g), w.numel(), lr, _stream(stream)))


def shadow_caps(B: int, fanout: int, hops: int):
    cn, ce = ctypes.c_int32(), ctypes.c_int64()
    _check(lib().gnn_shadow_caps(B, fanout, hops, ctypes.byref(cn), ctypes.byref(ce)))
    return int(cn.value), int(ce.value)


def sample_shadow(csr: Csr, roots: torch.Tensor, fanout: int, hops: int, rng_key: int, stream=None):
    """Returns (union block, comp_ptr [B + 1], root-row block)."""
    B = int(roots.shape[0])
    dev = roots.device
    cn, ce = shadow_caps(B, fanout, hops)
    kw = dict(dtype=torch.int32, device=dev)
    sub = Block(torch.zeros(cn + 1, **kw), torch.zeros(max(1, ce), **kw), torch.zeros(max(1, cn), **kw),
                torch.zeros(max(1, cn), **kw), torch.zeros(4, **kw), cn, cn, ce)
    comp_ptr = torch.zeros(B + 1, **kw)
    ro_counts = torch.zeros(4, **kw)
    wsb = int(lib().gnn_shadow_workspace_bytes(B, fanout, hops))
    ws = torch.empty(max(1, wsb), dtype=torch.uint8, device=dev)
    cb = sub.cstruct()
    _check(lib().gnn_sample_shadow(ctypes.byref(csr.c), _ptr(roots), B, fanout, hops, rng_key,
                                   ctypes.byref(cb), _ptr(comp_ptr), _ptr(ro_counts), _ptr(ws), wsb,
                                   _stream(stream)))
    ro = Block(sub.indptr, sub.indices, sub.src_nodes, sub.src_occ, ro_counts, B, cn, ce)
    return sub, comp_ptr, ro


def check_errors(stream=None) -> int:
    bits = ctypes.c_int32(0)
    rc = lib().gnn_check_errors(_stream(stream), ctypes.byref(bits))
    if rc not in (OK, EDEVICE):
        _check(rc)
    return int(bits.value)


# ---------------------------------------------------------------------------
# dynamic load balancing
# ---------------------------------------------------------------------------
def _model_struct(kind: str | int, dims: Sequence[int]) -> CModel:
    k = KIND[kind] if isinstance(kind, str) else int(kind)
    d = [int(x) for x in dims]
    cdims = (ctypes.c_int32 * (MAX_LAYERS + 1))(*(d + [0] * (MAX_LAYERS + 1 - len(d))))
    return CModel(k, len(d) - 1, cdims, None)


def estimate_work(csr: Csr, kind: str | int, dims: Sequence[int], batches, B: int,
                  fanouts: Optional[Sequence[int]] = None, shadow: Optional[tuple] = None,
                  ws: Optional[torch.Tensor] = None, stream=None):
    """Workload estimate of every batch (gnn_estimate_work, or with shadow =
    (fanout, hops) gnn_shadow_estimate_work).  batches: [(ids, rng_key)] with
    ids device int32 [B].  Returns device int64 tensors (work [n], edges
    [n x L] or [n x 2]); valid once the stream reaches this point."""
    m = _model_struct(kind, dims)
    L = len(dims) - 1
    n = len(batches)
    dev = batches[0][0].device if n else torch.device("cuda")
    ids = (ctypes.c_void_p * max(1, n))(*[_ptr(b[0]) for b in batches])
    keys = (ctypes.c_uint64 * max(1, n))(*[int(b[1]) for b in batches])
    if shadow is None:
        wsb = int(lib().gnn_estimate_workspace_bytes(B, _i32arr(fanouts), L, csr.num_nodes))
        cols = L
    else:
        wsb = int(lib().gnn_shadow_estimate_workspace_bytes(B, shadow[0], shadow[1]))
        cols = 2
    if wsb == 0:
        raise GnnError(EINVAL, "estimate_work: bad sizes")
    if ws is None or ws.numel() < wsb:
        ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    work = torch.zeros(max(1, n), dtype=torch.int64, device=dev)
    edges = torch.zeros((max(1, n), cols), dtype=torch.int64, device=dev)
    if shadow is None:
        _check(lib().gnn_estimate_work(ctypes.byref(m), ctypes.byref(csr.c), ids, keys, n, B,
                                       _i32arr(fanouts), _ptr(work), _ptr(edges), _ptr(ws), wsb,
                                       _stream(stream)))
    else:
        _check(lib().gnn_shadow_estimate_work(ctypes.byref(m), ctypes.byref(csr.c), ids, keys, n, B,
                                              shadow[0], shadow[1], _ptr(work), _ptr(edges),
                                              _ptr(ws), wsb, _stream(stream)))
    return work[:n], edges[:n]


def dlb_assign(work: Sequence[int], ratio: Sequence[float]):
    """(worker ids [n], load per worker [k]) of gnn_dlb_assign (host only)."""
    n, k = len(work), len(ratio)
    w = (ctypes.c_int64 * max(1, n))(*[int(x) for x in work])
    r = (ctypes.c_double * k)(*[float(x) for x in ratio])
    out = (ctypes.c_int32 * max(1, n))()
    load = (ctypes.c_int64 * k)()
    _check(lib().gnn_dlb_assign(w, n, r, k, out, load))
    return list(out)[:n], list(load)


def dlb_ratio(load: Sequence[int], seconds: Sequence[float], prev: Sequence[float],
              tolerance: float) -> List[float]:
    """Next ratio of gnn_dlb_ratio (host only)."""
    k = len(prev)
    ld = (ctypes.c_int64 * k)(*[int(x) for x in load])
    sec = (ctypes.c_double * k)(*[float(x) for x in seconds])
    pr = (ctypes.c_double * k)(*[float(x) for x in prev])
    out = (ctypes.c_double * k)()
    _check(lib().gnn_dlb_ratio(ld, sec, pr, k, float(tolerance), out))
    return list(out)


# ---------------------------------------------------------------------------
# GPU feature cache of a host-resident feature table
# ---------------------------------------------------------------------------
class FeatureCache:
    """A set-associative LRU cache in device memory (gnn_feature_cache_*)."""

    def __init__(self, num_sets: int, ways: int, width: int, dtype: int = F32, device="cuda"):
        nbytes = int(lib().gnn_feature_cache_bytes(num_sets, ways, width, dtype))
        if nbytes == 0:
            raise GnnError(EINVAL, "FeatureCache: bad sizes")
        # 256-byte aligned: torch's allocator hands out 512-byte aligned blocks
        self.mem = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.c = CFeatureCache(num_sets, ways, width, dtype, self.mem.data_ptr())
        self.num_sets, self.ways, self.width, self.dtype = num_sets, ways, width, dtype
        self._ws = None
        self.reset()

    def reset(self, stream=None):
        _check(lib().gnn_feature_cache_reset(ctypes.byref(self.c), _stream(stream)))

    def views(self):
        """(keys [S x W] int32, stamps [S x W] int32 bit patterns of uint32) as tensors."""
        k, st, r = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_void_p()
        _check(lib().gnn_feature_cache_views(ctypes.byref(self.c), ctypes.byref(k), ctypes.byref(st),
                                             ctypes.byref(r)))
        n = self.num_sets * self.ways
        keys = ws_view(self.mem, k.value, n, torch.int32).reshape(self.num_sets, self.ways)
        stamps = ws_view(self.mem, st.value, n, torch.int32).reshape(self.num_sets, self.ways)
        return keys, stamps

    def gather(self, X: torch.Tensor, ids: torch.Tensor, n_ids: torch.Tensor, cap: int,
               stats: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
        """out[i] = X[ids[i]] for i < min(*n_ids, cap) through the cache.  X may be
        pinned host memory.  stats: device int64 [2] += (hits, misses)."""
        if out is None:
            out = torch.empty((max(1, cap), self.width), dtype=X.dtype, device=self.mem.device)
        wsb = int(lib().gnn_gather_cached_workspace_bytes(self.num_sets, cap))
        if self._ws is None or self._ws.numel() < wsb:
            self._ws = torch.empty(max(1, wsb), dtype=torch.uint8, device=self.mem.device)
        _check(lib().gnn_gather_cached(ctypes.byref(self.c), _ptr(X), X.shape[0], X.stride(0),
                                       _ptr(ids), _ptr(n_ids), cap, _ptr(out), out.stride(0),
                                       _ptr(stats), _ptr(self._ws), wsb, _stream(stream)))
        return out


# ---------------------------------------------------------------------------
# training step
# ---------------------------------------------------------------------------
class Trainer:
    """Owns the weights and the step workspace of one model on one device."""

    def __init__(self, kind: str | int, dims: Sequence[int], weights: Sequence[torch.Tensor] | torch.Tensor,
                 B: int, fanouts: Sequence[int], num_nodes: int, x_dtype: int = F32,
                 device="cuda", shadow: Optional[tuple] = None, cache_sets: Optional[int] = None,
                 optimizer: str = "sgd", betas=(0.9, 0.999), eps: float = 1e-8):
        """shadow: None for neighbour sampling with `fanouts`, or (fanout, hops) for
        ShaDow subgraphs (then `fanouts` is ignored).  cache_sets: the set count of
        the FeatureCache that step_cached will use (sizes the workspace).
        optimizer: "sgd" (default) or "adam" (betas, eps; moments kept in
        self.adam_m / self.adam_v, steps taken in self.opt.steps)."""
        self.kind = KIND[kind] if isinstance(kind, str) else int(kind)
        self.dims = [int(d) for d in dims]
        self.B, self.fanouts, self.N, self.x_dtype = int(B), list(fanouts), int(num_nodes), x_dtype
        L = len(self.dims) - 1
        cdims = (ctypes.c_int32 * (MAX_LAYERS + 1))(*(self.dims + [0] * (MAX_LAYERS + 1 - len(self.dims))))
        self.model = CModel(self.kind, L, cdims, None)
        n = int(lib().gnn_num_params(ctypes.byref(self.model)))
        if isinstance(weights, torch.Tensor):
            flat = weights.to(device=device, dtype=torch.float32).contiguous().reshape(-1)
        else:
            flat = torch.cat([torch.as_tensor(w).reshape(-1).float() for w in weights]).to(device)
        assert flat.numel() == n, (flat.numel(), n)
        self.weights = flat.contiguous()
        self.model.weights = self.weights.data_ptr()
        self.opt = None
        if optimizer == "adam":
            self.adam_m = torch.zeros(n, dtype=torch.float32, device=device)
            self.adam_v = torch.zeros(n, dtype=torch.float32, device=device)
            self.opt = COptimizer(OPT_ADAM, float(betas[0]), float(betas[1]), float(eps),
                                  self.adam_m.data_ptr(), self.adam_v.data_ptr(), 0)
            self.model.opt = ctypes.pointer(self.opt)
        elif optimizer != "sgd":
            raise GnnError(EINVAL, f"unknown optimizer {optimizer}")
        self.shadow = tuple(shadow) if shadow else None
        if self.shadow:
            self.ws_bytes = int(lib().gnn_shadow_train_workspace_bytes(
                ctypes.byref(self.model), x_dtype, self.B, self.shadow[0], self.shadow[1]))
        elif cache_sets:
            self.ws_bytes = int(lib().gnn_train_cached_workspace_bytes(
                ctypes.byref(self.model), x_dtype, self.B, _i32arr(self.fanouts), self.N, cache_sets))
        else:
            self.ws_bytes = int(lib().gnn_train_workspace_bytes(ctypes.byref(self.model), x_dtype,
                                                                self.B, _i32arr(self.fanouts), self.N))
        if self.ws_bytes == 0:
            raise GnnError(EINVAL, lib().gnn_last_error().decode())
        self.ws = torch.zeros(self.ws_bytes, dtype=torch.uint8, device=device)
        self.loss = torch.zeros(1, dtype=torch.float32, device=device)
        self.device = device

    def step(self, csr: Csr, X: torch.Tensor, labels: torch.Tensor, seeds: torch.Tensor,
             rng_key: int, lr: float, stream=None, events=None):
        """One training step; `events` is None or a ctypes array of 2 * NUM_STAGES hipEvent_t."""
        assert seeds.dtype == torch.int32 and seeds.numel() == self.B
        if self.shadow:
            _check(lib().gnn_shadow_train_step(ctypes.byref(self.model), ctypes.byref(csr.c), _ptr(X),
                                               self.x_dtype, X.stride(0), _ptr(labels), _ptr(seeds),
                                               self.B, self.shadow[0], self.shadow[1], rng_key, lr,
                                               _ptr(self.loss), _ptr(self.ws), self.ws_bytes, events,
                                               _stream(stream)))
        else:
            _check(lib().gnn_train_step_ex(ctypes.byref(self.model), ctypes.byref(csr.c), _ptr(X),
                                           self.x_dtype, X.stride(0), _ptr(labels), _ptr(seeds),
                                           self.B, _i32arr(self.fanouts), rng_key, lr,
                                           _ptr(self.loss), _ptr(self.ws), self.ws_bytes, events,
                                           _stream(stream)))
        return self.loss

    def step_cached(self, csr: Csr, X: torch.Tensor, cache: "FeatureCache", stats: torch.Tensor,
                    labels: torch.Tensor, seeds: torch.Tensor, rng_key: int, lr: float, stream=None):
        """A training step whose feature table X stays in host memory (pinned):
        layer 1's rows are fetched through `cache` (stats: device int64 [2] +=
        (hits, misses)).  Needs cache_sets at construction."""
        assert seeds.dtype == torch.int32 and seeds.numel() == self.B and not self.shadow
        _check(lib().gnn_train_step_cached(ctypes.byref(self.model), ctypes.byref(csr.c), _ptr(X),
                                           self.x_dtype, X.stride(0), ctypes.byref(cache.c),
                                           _ptr(stats), _ptr(labels), _ptr(seeds), self.B,
                                           _i32arr(self.fanouts), rng_key, lr, _ptr(self.loss),
                                           _ptr(self.ws), self.ws_bytes, _stream(stream)))
        return self.loss

    def sample(self, csr: Csr, X: torch.Tensor, seeds: torch.Tensor, rng_key: int, slot: int,
               stream=None):
        """The sampling part of a step for `seeds` (and layer 1's aggregation of X),
        into block slot `slot` (0 or 1)."""
        assert seeds.dtype == torch.int32 and seeds.numel() == self.B
        if self.shadow:
            _check(lib().gnn_shadow_train_sample(ctypes.byref(self.model), ctypes.byref(csr.c), _ptr(X),
                                                 self.x_dtype, X.stride(0), _ptr(seeds), self.B,
                                                 self.shadow[0], self.shadow[1], rng_key, _ptr(self.ws),
                                                 self.ws_bytes, slot, _stream(stream)))
        else:
            _check(lib().gnn_train_sample(ctypes.byref(self.model), ctypes.byref(csr.c), _ptr(X),
                                          self.x_dtype, X.stride(0), _ptr(seeds), self.B,
                                          _i32arr(self.fanouts), rng_key, _ptr(self.ws), self.ws_bytes,
                                          slot, _stream(stream)))

    def model_pass(self, csr: Csr, X: torch.Tensor, labels: torch.Tensor, seeds: torch.Tensor,
                   lr: float, slot: int, stream=None, events=None):
        """The rest of a step (features, layers, loss, backward, SGD) on block slot `slot`."""
        assert seeds.dtype == torch.int32 and seeds.numel() == self.B
        if self.shadow:
            _check(lib().gnn_shadow_train_model(ctypes.byref(self.model), ctypes.byref(csr.c), _ptr(X),
                                                self.x_dtype, X.stride(0), _ptr(labels), _ptr(seeds),
                                                self.B, self.shadow[0], self.shadow[1], lr,
                                                _ptr(self.loss), _ptr(self.ws), self.ws_bytes, slot,
                                                events, _stream(stream)))
        else:
            _check(lib().gnn_train_model(ctypes.byref(self.model), ctypes.byref(csr.c), _ptr(X),
                                         self.x_dtype, X.stride(0), _ptr(labels), _ptr(seeds), self.B,
                                         _i32arr(self.fanouts), lr, _ptr(self.loss), _ptr(self.ws),
                                         self.ws_bytes, slot, events, _stream(stream)))
        return self.loss

    def run_pipelined(self, csr: Csr, X: torch.Tensor, labels: torch.Tensor, batches, lr: float,
                      model_stream=None, sample_stream=None) -> torch.Tensor:
        """Train on `batches` (a sequence of (seeds, rng_key)) with one library call
        (gnn_train_pipelined): batch i + 1 is sampled on `sample_stream` while batch i
        trains on `model_stream` (default-priority torch streams; defaults: the current
        stream and a stream kept by the trainer).  Returns a device tensor of the n
        losses (loss of step i before its update); no host sync."""
        n = len(batches)
        losses = torch.zeros(max(1, n), dtype=torch.float32, device=self.device)
        if n == 0:
            return losses[:0]
        ms = model_stream if model_stream is not None else torch.cuda.current_stream()
        if sample_stream is None:
            if getattr(self, "_sample_stream", None) is None:
                self._sample_stream = torch.cuda.Stream(device=self.device)
            sample_stream = self._sample_stream
        if getattr(self, "_events", None) is None:
            self._events = _HipEvents(4)
        for seeds, _ in batches:
            assert seeds.dtype == torch.int32 and seeds.numel() == self.B
        sp = (ctypes.c_void_p * n)(*[s.data_ptr() for s, _ in batches])
        keys = (ctypes.c_uint64 * n)(*[int(k) for _, k in batches])
        if self.shadow:
            _check(lib().gnn_shadow_train_pipelined(
                ctypes.byref(self.model), ctypes.byref(csr.c), _ptr(X), self.x_dtype, X.stride(0),
                _ptr(labels), sp, keys, n, self.B, self.shadow[0], self.shadow[1], lr, _ptr(losses),
                _ptr(self.ws), self.ws_bytes, self._events.array, _stream(ms), _stream(sample_stream)))
        else:
            _check(lib().gnn_train_pipelined(
                ctypes.byref(self.model), ctypes.byref(csr.c), _ptr(X), self.x_dtype, X.stride(0),
                _ptr(labels), sp, keys, n, self.B, _i32arr(self.fanouts), lr, _ptr(losses),
                _ptr(self.ws), self.ws_bytes, self._events.array, _stream(ms), _stream(sample_stream)))
        # the batches' seed tensors and the loss array stay alive until the streams finish
        self._inflight = (batches, losses)
        return losses

    def views(self, slot: int = 0) -> CTrainViews:
        """Where the workspace keeps the step's intermediates; `slot` selects the
        block slot (neighbour sampling; ShaDow views slot 0)."""
        v = CTrainViews()
        if self.shadow:
            assert slot == 0
            _check(lib().gnn_shadow_train_step_views(ctypes.byref(self.model), self.x_dtype, self.B,
                                                     self.shadow[0], self.shadow[1], _ptr(self.ws),
                                                     self.ws_bytes, ctypes.byref(v)))
        else:
            _check(lib().gnn_train_slot_views(ctypes.byref(self.model), self.x_dtype, self.B,
                                              _i32arr(self.fanouts), self.N, _ptr(self.ws),
                                              self.ws_bytes, slot, ctypes.byref(v)))
        return v

    def inspect(self, slot: int = 0):
        """Host copies of the last step's intermediates (after synchronising).
        With pipelined steps, `slot` picks the block slot whose blocks and
        layer-1 GEMM input are returned (step i uses slot i mod 2); the other
        entries hold the last model pass."""
        torch.cuda.synchronize()
        v = self.views(slot)
        L = len(self.dims) - 1
        out = {}
        if self.shadow:
            blocks = [Block.from_ws(v.blocks[h], self.ws).host() for h in range(2)]
            out["comp_ptr"] = ws_view(self.ws, v.comp_ptr, self.B + 1, torch.int32).cpu().numpy()
            layer_block = [0] * (L - 1) + [1]      # layer l -> index into blocks
            n_src_outer = blocks[0][1]
        else:
            blocks = [Block.from_ws(v.blocks[h], self.ws).host() for h in range(L)]
            layer_block = [L - l for l in range(1, L + 1)]
            n_src_outer = blocks[L - 1][1]
        out["blocks"] = blocks
        # the step keeps no gathered feature copy (layer 1 reads X in place)
        out["xg"] = None
        if v.xg:
            xdt = torch.float32 if self.x_dtype == F32 else torch.int16
            out["xg"] = ws_view(self.ws, v.xg, n_src_outer * self.dims[0], xdt).reshape(
                n_src_outer, self.dims[0]).cpu()
        xs, hs = [], []
        for l in range(1, L + 1):
            nd = blocks[layer_block[l - 1]][0]
            w = int(v.x_ld[l - 1])
            if not v.x[l - 1]:   # GAT keeps layer 1's input rows only
                xs.append(None)
            elif v.x_dtype[l - 1] == BF16:  # widened exactly
                xs.append(ws_view(self.ws, v.x[l - 1], nd * w, torch.bfloat16).reshape(nd, w)
                          .float().cpu().numpy())
            else:
                xs.append(ws_view(self.ws, v.x[l - 1], nd * w, torch.float32).reshape(nd, w).cpu().numpy())
            hs.append(ws_view(self.ws, v.h[l - 1], nd * self.dims[l], torch.float32)
                      .reshape(nd, self.dims[l]).cpu().numpy())
        out["x"], out["h"] = xs, hs
        n = self.weights.numel()
        out["dweights"] = ws_view(self.ws, v.dweights, n, torch.float32).cpu().numpy()
        out["dlogits"] = ws_view(self.ws, v.dlogits, self.B * self.dims[L], torch.float32).reshape(
            self.B, self.dims[L]).cpu().numpy()
        return out


class Trace:
    """gnn_trace over caller-owned HIP events (handles as ints): while
    installed with `with trace:`, the i-th recorded launch of the library on
    this thread stamps its kernel's start and end into events[2 i] and
    events[2 i + 1]; names() lists the recorded kernels."""

    def __init__(self, events: Sequence[int], only: Optional[str] = None):
        assert len(events) % 2 == 0
        cap = len(events) // 2
        self._ev = (ctypes.c_void_p * max(1, len(events)))(*events)
        self._names = (ctypes.c_char_p * max(1, cap))()
        self._only = only.encode() if only else None
        self.c = CTrace(ctypes.cast(self._ev, ctypes.c_void_p), ctypes.cast(self._names, ctypes.c_void_p),
                        self._only, cap, 0, 0)

    def __enter__(self):
        _check(lib().gnn_trace_begin(ctypes.byref(self.c)))
        return self

    def __exit__(self, *exc):
        lib().gnn_trace_begin(None)
        return False

    @property
    def count(self) -> int:
        return int(self.c.count)

    @property
    def dropped(self) -> int:
        return int(self.c.dropped)

    def names(self) -> List[str]:
        return [self._names[i].decode() for i in range(self.count)]

    def reset(self):
        self.c.count = 0
        self.c.dropped = 0

