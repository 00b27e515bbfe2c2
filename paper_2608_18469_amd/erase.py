"""Python binding of liberase.so (the C ABI in include/erase.h).

Argument marshalling only: every step of the training path runs in the HIP
kernels behind the C ABI.  PyTorch is used for device memory
(``tensor.data_ptr()``) and streams (``torch.cuda.Stream().cuda_stream``).
There is no fallback: if the library is missing or no GPU is present, the
constructors raise.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_float, c_int32, c_int64, c_size_t, c_void_p

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liberase.so")

OK = 0
ERR_INVALID_ARG, ERR_SHAPE, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_STATE, ERR_NONFINITE = range(-1, -8, -1)
F32, BF16 = 0, 1
LINEAR_RELU, CROSS = 0, 1
LOSS_BCE = 0
IN_X, IN_PREV = 0, 1
SERIAL, OVERLAP, SERIAL_GRAPH, OVERLAP_GRAPH, PIPELINE, OVERLAP_ADAM_END, UNDETACHED, UNDETACHED_GRAPH = range(8)
SCHEDULES = {"serial": SERIAL, "overlap": OVERLAP, "serial_graph": SERIAL_GRAPH, "overlap_graph": OVERLAP_GRAPH,
             "pipeline": PIPELINE, "overlap_adam_end": OVERLAP_ADAM_END, "undetached": UNDETACHED,
             "undetached_graph": UNDETACHED_GRAPH}
DISPATCH_CALLER, DISPATCH_WORKER = 0, 1
DISPATCH = {"caller": DISPATCH_CALLER, "worker": DISPATCH_WORKER}
KERNEL_KINDS = {0: "prologue", 1: "fwd_gemm", 2: "head_bce", 3: "wgrad_gemm", 4: "dgrad_gemm", 5: "adam",
                6: "bwd_gemm", 7: "empty", 8: "fwd_head_gemm", 9: "fwd_gemm_kg2",
                10: "wgrad_gemm_kg2", 11: "wgrad_adam_kg2"}


class LayerSpec(ctypes.Structure):
    _fields_ = [("kind", c_int32), ("in_dim", c_int32), ("out_dim", c_int32)]


class BlockSpec(ctypes.Structure):
    _fields_ = [("input_src", c_int32), ("n_layers", c_int32), ("layers", POINTER(LayerSpec)),
                ("loss", c_int32), ("lam", c_float)]


class Config(ctypes.Structure):
    _fields_ = [("n_blocks", c_int32), ("blocks", POINTER(BlockSpec)), ("batch", c_int32), ("in_dim", c_int32),
                ("x_ld", c_int32), ("dtype", c_int32), ("lr", c_float), ("beta1", c_float), ("beta2", c_float),
                ("eps", c_float), ("x_in_place", c_int32)]


class BlockBuffers(ctypes.Structure):
    _fields_ = [("param", c_void_p), ("m", c_void_p), ("v", c_void_p), ("grad", c_void_p)]


class KernelTime(ctypes.Structure):
    _fields_ = [("kind", c_int32), ("block", c_int32), ("layer", c_int32), ("stream", c_int32),
                ("start_ms", c_float), ("end_ms", c_float), ("tile_m", c_int32), ("tile_n", c_int32),
                ("split", c_int32), ("grid", c_int32), ("flops", c_double), ("bytes", c_double)]


# every entry point of include/erase.h with its ctypes signature
class BagConfig(ctypes.Structure):
    """erase_bag_config: shape of the embedding-bag input stage."""
    _fields_ = [("batch", c_int32), ("n_dense", c_int32), ("n_tables", c_int32), ("dim", c_int32),
                ("rows", c_int64), ("nnz", c_int64), ("dtype", c_int32), ("x_ld", c_int64)]


SIGNATURES = {
    "erase_param_count": (c_int32, [POINTER(Config), c_int32, POINTER(c_int64)]),
    "erase_workspace_bytes": (c_int32, [POINTER(Config), POINTER(c_size_t)]),
    "erase_init": (c_int32, [POINTER(Config), POINTER(BlockBuffers), c_void_p, c_size_t, c_void_p, c_void_p,
                             POINTER(c_void_p)]),
    "erase_init_streams": (c_int32, [POINTER(Config), POINTER(BlockBuffers), c_void_p, c_size_t, c_void_p,
                                     POINTER(c_void_p), c_int32, POINTER(c_void_p)]),
    "erase_step": (c_int32, [c_void_p, c_void_p, c_void_p, c_int32, c_void_p]),
    "erase_sync": (c_int32, [c_void_p]),
    "erase_get_step": (c_int32, [c_void_p, POINTER(c_int64)]),
    "erase_set_step": (c_int32, [c_void_p, c_int64]),
    "erase_refresh_weights": (c_int32, [c_void_p]),
    "erase_set_timing": (c_int32, [c_void_p, c_int32]),
    "erase_set_dispatch": (c_int32, [c_void_p, c_int32]),
    "erase_embed_bags": (c_int32, [POINTER(BagConfig), c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                   c_void_p]),
    "erase_embed_bags_backward_scratch_bytes": (c_int32, [POINTER(BagConfig), POINTER(c_size_t)]),
    "erase_embed_bags_backward": (c_int32, [POINTER(BagConfig), c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                            c_size_t, c_void_p, c_void_p]),
    "erase_embed_bags_backward_noalloc": (c_int32, [POINTER(BagConfig), c_void_p, c_void_p, c_void_p, c_void_p,
                                                    c_void_p, c_void_p]),
    "erase_read_timing": (c_int32, [c_void_p, POINTER(KernelTime), c_int32, POINTER(c_int32)]),
    "erase_destroy": (c_int32, [c_void_p]),
    "erase_status_str": (ctypes.c_char_p, [c_int32]),
    "erase_last_error": (ctypes.c_char_p, [c_void_p]),
}

_lib = None


def lib() -> ctypes.CDLL:
    """Load liberase.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_18469_amd.build` "
                               "(or __graft_entry__.build()); there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


class EraseError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        msg = lib().erase_status_str(status).decode()
        super().__init__(f"{where}: {msg} ({status}){': ' + detail if detail else ''}")
        self.status = status


def _check(status: int, where: str, ctx=None):
    if status != OK:
        detail = lib().erase_last_error(ctx).decode() if ctx else ""
        raise EraseError(status, where, detail)


class NativeConfig:
    """ctypes view of a model description (see ``synth.config``), kept alive
    together with the arrays it points to."""

    def __init__(self, cfg: dict, x_ld: int | None = None, x_in_place: bool = False):
        esz = 2 if cfg["dtype"] == "bf16" else 4
        per16 = 16 // esz
        if x_ld is None:
            x_ld = (cfg["in_dim"] + per16 - 1) // per16 * per16
        self.x_ld = int(x_ld)
        self._layers = []
        blocks = (BlockSpec * len(cfg["blocks"]))()
        for i, blk in enumerate(cfg["blocks"]):
            arr = (LayerSpec * len(blk["layers"]))()
            for j, (kind, fin, fout) in enumerate(blk["layers"]):
                arr[j] = LayerSpec(LINEAR_RELU if kind == "linear_relu" else CROSS, fin, fout)
            self._layers.append(arr)
            blocks[i] = BlockSpec(IN_X if blk["input"] == "x" else IN_PREV, len(blk["layers"]),
                                  ctypes.cast(arr, POINTER(LayerSpec)), LOSS_BCE, float(blk["lam"]))
        self._blocks = blocks
        ad = cfg["adam"]
        self.c = Config(len(cfg["blocks"]), ctypes.cast(blocks, POINTER(BlockSpec)), cfg["batch"], cfg["in_dim"],
                        self.x_ld, BF16 if cfg["dtype"] == "bf16" else F32, ad["lr"], ad["beta1"], ad["beta2"],
                        ad["eps"], 1 if x_in_place else 0)

    def ptr(self):
        return ctypes.byref(self.c)


def param_count(ncfg: NativeConfig, block: int) -> int:
    n = c_int64(0)
    _check(lib().erase_param_count(ncfg.ptr(), block, ctypes.byref(n)), "erase_param_count")
    return n.value


def workspace_bytes(ncfg: NativeConfig) -> int:
    n = c_size_t(0)
    _check(lib().erase_workspace_bytes(ncfg.ptr(), ctypes.byref(n)), "erase_workspace_bytes")
    return n.value


def pack_block(p: dict) -> np.ndarray:
    """Flat fp32 vector in the ABI order: per layer W[out][in], b; then w, c."""
    parts = []
    for (W, b) in p["layers"]:
        parts += [np.asarray(W, np.float32).reshape(-1), np.asarray(b, np.float32).reshape(-1)]
    parts += [np.asarray(p["head"][0], np.float32).reshape(-1), np.asarray(p["head"][1], np.float32).reshape(-1)]
    return np.concatenate(parts)


def unpack_block(blk: dict, flat: np.ndarray) -> dict:
    off = 0
    layers = []
    for (_k, fin, fout) in blk["layers"]:
        W = flat[off:off + fin * fout].reshape(fout, fin)
        off += fin * fout
        b = flat[off:off + fout]
        off += fout
        layers.append((W, b))
    last = blk["layers"][-1][2]
    w = flat[off:off + last]
    off += last
    c = flat[off:off + 1]
    off += 1
    assert off == flat.size
    return {"layers": layers, "head": (w, c)}


def embed_bags(dense, offsets, indices, tables, x, status=None, stream=None):
    """The embedding-bag input stage (erase_embed_bags) on device tensors:
    dense fp32 [M][n_dense] (or None), offsets int64 [T][M+1], indices int32
    [nnz], tables fp32 [T][rows][dim], x [M][x_ld] float32 or bfloat16 (the
    output), status int32 [1] or None.  Enqueued on `stream` (a torch stream;
    default: the current one); returns without waiting."""
    import torch
    M, x_ld = x.shape
    T, rows, dim = tables.shape
    n_dense = 0 if dense is None else dense.shape[1]
    for name, t, dt in (("offsets", offsets, torch.int64), ("indices", indices, torch.int32),
                        ("tables", tables, torch.float32)):
        if t.dtype != dt or not t.is_contiguous():
            raise EraseError(ERR_INVALID_ARG, "embed_bags", f"{name} must be a contiguous {dt} tensor")
    if dense is not None and (dense.dtype != torch.float32 or not dense.is_contiguous()):
        raise EraseError(ERR_INVALID_ARG, "embed_bags", "dense must be a contiguous float32 tensor")
    if x.dtype not in (torch.float32, torch.bfloat16) or x.stride(1) != 1:
        raise EraseError(ERR_INVALID_ARG, "embed_bags", "x must be float32 or bfloat16 with unit column stride")
    if tuple(offsets.shape) != (T, M + 1):
        raise EraseError(ERR_SHAPE, "embed_bags", "offsets must be [n_tables][batch + 1]")
    cfg = BagConfig(M, n_dense, T, dim, rows, indices.numel(), BF16 if x.dtype == torch.bfloat16 else F32,
                    x.stride(0))
    s = (stream or torch.cuda.current_stream()).cuda_stream
    ptr = (lambda t: None if t is None or t.numel() == 0 else t.data_ptr())
    _check(lib().erase_embed_bags(ctypes.byref(cfg), ptr(dense), offsets.data_ptr(), ptr(indices),
                                  tables.data_ptr(), x.data_ptr(), ptr(status), s), "erase_embed_bags")


def embed_bags_backward(offsets, indices, dx, n_dense, rows, dim, table_grad=None, status=None, stream=None):
    """Backward of the embedding-bag stage (erase_embed_bags_backward) on device
    tensors: offsets int64 [T][M+1], indices int32 [nnz], dx [M][x_ld] float32
    or bfloat16 (the gradient at x), n_dense, rows, dim as in the forward.
    Returns table_grad fp32 [T][rows][dim] (allocated unless given) and
    allocates the scratch; enqueued on `stream` (default: the current one)."""
    import torch
    T = offsets.shape[0]
    M, x_ld = dx.shape
    for name, t, dt in (("offsets", offsets, torch.int64), ("indices", indices, torch.int32)):
        if t.dtype != dt or not t.is_contiguous():
            raise EraseError(ERR_INVALID_ARG, "embed_bags_backward", f"{name} must be a contiguous {dt} tensor")
    if dx.dtype not in (torch.float32, torch.bfloat16) or dx.stride(1) != 1:
        raise EraseError(ERR_INVALID_ARG, "embed_bags_backward", "dx must be float32 or bfloat16, unit column stride")
    cfg = BagConfig(M, n_dense, T, dim, rows, indices.numel(), BF16 if dx.dtype == torch.bfloat16 else F32,
                    dx.stride(0))
    need = c_size_t(0)
    _check(lib().erase_embed_bags_backward_scratch_bytes(ctypes.byref(cfg), ctypes.byref(need)),
           "erase_embed_bags_backward_scratch_bytes")
    scratch = torch.empty(need.value, dtype=torch.uint8, device=dx.device)
    if table_grad is None:
        table_grad = torch.empty((T, rows, dim), dtype=torch.float32, device=dx.device)
    s = (stream or torch.cuda.current_stream()).cuda_stream
    ptr = (lambda t: None if t is None or t.numel() == 0 else t.data_ptr())
    _check(lib().erase_embed_bags_backward(ctypes.byref(cfg), offsets.data_ptr(), ptr(indices), dx.data_ptr(),
                                           table_grad.data_ptr(), scratch.data_ptr(), need.value, ptr(status), s),
           "erase_embed_bags_backward")
    return table_grad, scratch


BAG_SCRATCH_MAX = 64 << 20  # ERASE_BAG_SCRATCH_MAX of include/erase.h


def embed_bags_backward_noalloc(offsets, indices, dx, n_dense, rows, dim, table_grad, status=None, stream=None):
    """erase_embed_bags_backward_noalloc: the backward of the embedding-bag
    stage with the library's static device scratch (for callers that cannot
    allocate); arguments as for embed_bags_backward, table_grad given.  Calls
    that overlap on one GPU share the scratch and race."""
    import torch
    T = offsets.shape[0]
    M, x_ld = dx.shape
    for name, t, dt in (("offsets", offsets, torch.int64), ("indices", indices, torch.int32),
                        ("table_grad", table_grad, torch.float32)):
        if t.dtype != dt or not t.is_contiguous():
            raise EraseError(ERR_INVALID_ARG, "embed_bags_backward_noalloc", f"{name} must be a contiguous {dt} tensor")
    if dx.dtype not in (torch.float32, torch.bfloat16) or dx.stride(1) != 1:
        raise EraseError(ERR_INVALID_ARG, "embed_bags_backward_noalloc",
                         "dx must be float32 or bfloat16, unit column stride")
    cfg = BagConfig(M, n_dense, T, dim, rows, indices.numel(), BF16 if dx.dtype == torch.bfloat16 else F32,
                    dx.stride(0))
    s = (stream or torch.cuda.current_stream()).cuda_stream
    ptr = (lambda t: None if t is None or t.numel() == 0 else t.data_ptr())
    _check(lib().erase_embed_bags_backward_noalloc(ctypes.byref(cfg), offsets.data_ptr(), ptr(indices),
                                                   dx.data_ptr(), table_grad.data_ptr(), ptr(status), s),
           "erase_embed_bags_backward_noalloc")
    return table_grad


class Trainer:
    """Owns the device buffers, two streams and one library context."""

    def __init__(self, cfg: dict, params: list, x_ld: int | None = None, keep_grads: bool = True,
                 m: list | None = None, v: list | None = None, step: int = 0, bwd_streams: int = 1,
                 streams=None, x_in_place: bool = False):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("no HIP device available: the ERASE step runs only on the GPU")
        lib()
        self.torch = torch
        self.cfg = cfg
        self.dev = torch.device("cuda", torch.cuda.current_device())
        # x read in place: rows of a multiple of 128 elements (zero tails, as
        # device_batch and erase_embed_bags write them)
        if x_in_place and x_ld is None:
            x_ld = (cfg["in_dim"] + 127) // 128 * 128
        self.ncfg = NativeConfig(cfg, x_ld, x_in_place)
        self.act_dtype = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
        nb = len(cfg["blocks"])
        self.param, self.m, self.v, self.grad = [], [], [], []
        bufs = (BlockBuffers * nb)()
        for b in range(nb):
            n = param_count(self.ncfg, b)
            flat = pack_block(params[b])
            assert flat.size == n, (flat.size, n)
            P = torch.from_numpy(flat).to(self.dev)
            Mm = torch.from_numpy(pack_block(m[b])).to(self.dev) if m else torch.zeros(n, device=self.dev)
            Vv = torch.from_numpy(pack_block(v[b])).to(self.dev) if v else torch.zeros(n, device=self.dev)
            G = torch.zeros(n, device=self.dev) if keep_grads else None
            self.param.append(P); self.m.append(Mm); self.v.append(Vv); self.grad.append(G)
            bufs[b] = BlockBuffers(P.data_ptr(), Mm.data_ptr(), Vv.data_ptr(), G.data_ptr() if G is not None else None)
        self._bufs = bufs
        self.ws_bytes = workspace_bytes(self.ncfg)
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=self.dev)
        pad = (-self.ws.data_ptr()) % 256
        self.ws_ptr = self.ws.data_ptr() + pad
        if streams is not None:
            # caller-owned streams (torch streams, or torch.cuda.ExternalStream
            # around HIP handles): (forward, [backward, ...])
            self.sf, self.sbs = streams[0], list(streams[1])
            bwd_streams = len(self.sbs)
        else:
            self.sf = torch.cuda.Stream(device=self.dev)
            self.sbs = [torch.cuda.Stream(device=self.dev) for _ in range(bwd_streams)]
        self.sb = self.sbs[0]
        torch.cuda.synchronize(self.dev)
        ctx = c_void_p()
        sb_arr = (c_void_p * bwd_streams)(*[s.cuda_stream for s in self.sbs])
        _check(lib().erase_init_streams(self.ncfg.ptr(), bufs, c_void_p(self.ws_ptr), self.ws_bytes,
                                        c_void_p(self.sf.cuda_stream), sb_arr, bwd_streams, ctypes.byref(ctx)),
               "erase_init_streams")
        self.ctx = ctx
        if step:
            self.set_step(step)
        self.losses = torch.zeros(nb, dtype=torch.float32, device=self.dev)

    # -- inputs ---------------------------------------------------------------
    def device_batch(self, x: np.ndarray, y: np.ndarray):
        """Copy one batch to the device in the ABI layout ([M][x_ld] of the
        activation dtype, fp32 labels)."""
        torch = self.torch
        M, K = x.shape
        xt = torch.zeros((M, self.ncfg.x_ld), dtype=self.act_dtype, device=self.dev)
        xt[:, :K] = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(self.dev).to(self.act_dtype)
        yt = torch.from_numpy(np.ascontiguousarray(y, dtype=np.float32)).to(self.dev)
        torch.cuda.synchronize(self.dev)
        return xt, yt

    # -- stepping -------------------------------------------------------------
    def step(self, x, y, schedule="overlap", losses=None, wait_current=True):
        """Enqueue one step on the library's streams (non-blocking)."""
        if wait_current:
            self.sf.wait_stream(self.torch.cuda.current_stream(self.dev))
        sched = SCHEDULES[schedule] if isinstance(schedule, str) else int(schedule)
        out = self.losses if losses is None else losses
        _check(lib().erase_step(self.ctx, c_void_p(x.data_ptr()), c_void_p(y.data_ptr()), sched,
                                c_void_p(out.data_ptr())), "erase_step", self.ctx)
        return out

    def sync(self):
        _check(lib().erase_sync(self.ctx), "erase_sync", self.ctx)

    def get_step(self) -> int:
        t = c_int64(0)
        _check(lib().erase_get_step(self.ctx, ctypes.byref(t)), "erase_get_step", self.ctx)
        return t.value

    def set_step(self, t: int):
        _check(lib().erase_set_step(self.ctx, int(t)), "erase_set_step", self.ctx)

    def refresh_weights(self):
        _check(lib().erase_refresh_weights(self.ctx), "erase_refresh_weights", self.ctx)

    def set_timing(self, on: bool):
        _check(lib().erase_set_timing(self.ctx, 1 if on else 0), "erase_set_timing", self.ctx)

    def set_dispatch(self, mode: str):
        """'caller' (every launch from the calling thread) or 'worker' (a
        library-owned host thread enqueues the backward streams' work of the
        ERASE schedules)."""
        _check(lib().erase_set_dispatch(self.ctx, DISPATCH[mode]), "erase_set_dispatch", self.ctx)

    def read_timing(self):
        n = c_int32(0)
        cap = 4096
        arr = (KernelTime * cap)()
        _check(lib().erase_read_timing(self.ctx, arr, cap, ctypes.byref(n)), "erase_read_timing", self.ctx)
        return [dict(kind=KERNEL_KINDS[a.kind], block=a.block, layer=a.layer, stream=a.stream,
                     start_ms=a.start_ms, end_ms=a.end_ms, tile_m=a.tile_m, tile_n=a.tile_n, split=a.split,
                     grid=a.grid, flops=a.flops, bytes=a.bytes)
                for a in arr[:min(n.value, cap)]]

    # -- state ----------------------------------------------------------------
    def state(self):
        """(params, m, v, grads) as structured numpy trees (synchronizes)."""
        self.sync()
        out = []
        for bufs in (self.param, self.m, self.v, self.grad):
            out.append([None if t is None else unpack_block(blk, t.detach().cpu().numpy())
                        for blk, t in zip(self.cfg["blocks"], bufs)])
        return tuple(out)

    def flat_state(self):
        self.sync()
        return ([t.detach().cpu().numpy().copy() for t in self.param],
                [t.detach().cpu().numpy().copy() for t in self.m],
                [t.detach().cpu().numpy().copy() for t in self.v],
                [None if t is None else t.detach().cpu().numpy().copy() for t in self.grad])

    def close(self):
        if getattr(self, "ctx", None):
            lib().erase_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
