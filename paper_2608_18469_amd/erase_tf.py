"""Python binding of the small-transformer entry points of liberase.so (the C
ABI in include/erase_tf.h).

Argument marshalling only: every step of the training path runs in the HIP
kernels behind the C ABI; PyTorch provides device memory and streams.  There
is no fallback: without the library or a GPU the constructor raises.
"""
from __future__ import annotations

import ctypes
from ctypes import POINTER, c_float, c_int32, c_int64, c_size_t, c_void_p

import numpy as np

from . import erase, synth_tf
from .erase import BlockBuffers, EraseError, KernelTime, OK

TF_KERNEL_KINDS = {0: "prologue", 1: "fwd_gemm", 3: "wgrad_gemm", 4: "dgrad_gemm", 5: "adam", 6: "bwd_gemm", 7: "empty",
                   11: "embed", 12: "rms_fwd", 13: "rms_bwd", 14: "attn_fwd", 15: "attn_bwd", 16: "head_norm",
                   17: "emb_grad"}
GEMM_NAMES = {0: "qkv", 1: "proj", 2: "mlp_up", 3: "mlp_down", 4: "vocab"}
SCHEDULES = {"serial": erase.SERIAL, "overlap": erase.OVERLAP}
TENSORS = {"a0": 0, "n1": 1, "qkv": 2, "o": 3, "a1": 4, "n2": 5, "u": 6, "g": 7, "z": 8, "hn": 9,
           "logits": 10, "lse": 11, "dqkv": 12, "dz": 13, "rowscale": 14, "hns": 15}


class TfConfig(ctypes.Structure):
    _fields_ = [("vocab", c_int32), ("d_model", c_int32), ("n_heads", c_int32), ("n_layers", c_int32),
                ("seq_len", c_int32), ("batch", c_int32), ("lr", c_float), ("beta1", c_float),
                ("beta2", c_float), ("eps", c_float), ("lam", c_float)]


SIGNATURES = {
    "erase_tf_param_count": (c_int32, [POINTER(TfConfig), c_int32, POINTER(c_int64)]),
    "erase_tf_workspace_bytes": (c_int32, [POINTER(TfConfig), POINTER(c_size_t)]),
    "erase_tf_init": (c_int32, [POINTER(TfConfig), POINTER(BlockBuffers), c_void_p, c_size_t, c_void_p, c_void_p,
                                POINTER(c_void_p)]),
    "erase_tf_step": (c_int32, [c_void_p, c_void_p, c_int32, c_void_p]),
    "erase_tf_sync": (c_int32, [c_void_p]),
    "erase_tf_get_step": (c_int32, [c_void_p, POINTER(c_int64)]),
    "erase_tf_set_step": (c_int32, [c_void_p, c_int64]),
    "erase_tf_refresh_weights": (c_int32, [c_void_p]),
    "erase_tf_set_timing": (c_int32, [c_void_p, c_int32]),
    "erase_tf_read_timing": (c_int32, [c_void_p, POINTER(KernelTime), c_int32, POINTER(c_int32)]),
    "erase_tf_tensor": (c_int32, [c_void_p, c_int32, c_int32, POINTER(c_void_p), POINTER(c_int64)]),
    "erase_tf_destroy": (c_int32, [c_void_p]),
    "erase_tf_last_error": (ctypes.c_char_p, [c_void_p]),
}

_bound = False


def lib() -> ctypes.CDLL:
    global _bound
    L = erase.lib()
    if not _bound:
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _bound = True
    return L


def _check(status: int, where: str, ctx=None):
    if status != OK:
        detail = lib().erase_tf_last_error(ctx).decode() if ctx else ""
        raise EraseError(status, where, detail)


def native_config(cfg: dict) -> TfConfig:
    ad = cfg["adam"]
    return TfConfig(cfg["vocab"], cfg["d"], cfg["heads"], cfg["layers"], cfg["seq"], cfg["batch"], ad["lr"],
                    ad["beta1"], ad["beta2"], ad["eps"], float(cfg.get("lam", 1.0)))


def param_count(cfg: dict, block: int) -> int:
    n = c_int64(0)
    nc = native_config(cfg)
    _check(lib().erase_tf_param_count(ctypes.byref(nc), block, ctypes.byref(n)), "erase_tf_param_count")
    return n.value


def workspace_bytes(cfg: dict) -> int:
    n = c_size_t(0)
    nc = native_config(cfg)
    _check(lib().erase_tf_workspace_bytes(ctypes.byref(nc), ctypes.byref(n)), "erase_tf_workspace_bytes")
    return n.value


class TfTrainer:
    """Owns the device buffers, two streams and one transformer context."""

    def __init__(self, cfg: dict, params: list, keep_grads: bool = True, m: list | None = None,
                 v: list | None = None, step: int = 0):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("no HIP device available: the ERASE step runs only on the GPU")
        lib()
        self.torch = torch
        self.cfg = cfg
        self.dev = torch.device("cuda", torch.cuda.current_device())
        self.nc = native_config(cfg)
        L = cfg["layers"]
        self.param, self.m, self.v, self.grad = [], [], [], []
        bufs = (BlockBuffers * L)()
        for b in range(L):
            n = param_count(cfg, b)
            flat = synth_tf.pack_block(cfg, b, params[b])
            assert flat.size == n, (flat.size, n)
            P = torch.from_numpy(flat).to(self.dev)
            Mm = (torch.from_numpy(synth_tf.pack_block(cfg, b, m[b])).to(self.dev) if m
                  else torch.zeros(n, device=self.dev))
            Vv = (torch.from_numpy(synth_tf.pack_block(cfg, b, v[b])).to(self.dev) if v
                  else torch.zeros(n, device=self.dev))
            G = torch.zeros(n, device=self.dev) if keep_grads else None
            self.param.append(P); self.m.append(Mm); self.v.append(Vv); self.grad.append(G)
            bufs[b] = BlockBuffers(P.data_ptr(), Mm.data_ptr(), Vv.data_ptr(), G.data_ptr() if G is not None else None)
        self._bufs = bufs
        self.ws_bytes = workspace_bytes(cfg)
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=self.dev)
        self.ws_ptr = self.ws.data_ptr() + (-self.ws.data_ptr()) % 256
        self.sf = torch.cuda.Stream(device=self.dev)
        self.sb = torch.cuda.Stream(device=self.dev)
        torch.cuda.synchronize(self.dev)
        ctx = c_void_p()
        _check(lib().erase_tf_init(ctypes.byref(self.nc), bufs, c_void_p(self.ws_ptr), self.ws_bytes,
                                   c_void_p(self.sf.cuda_stream), c_void_p(self.sb.cuda_stream), ctypes.byref(ctx)),
               "erase_tf_init")
        self.ctx = ctx
        if step:
            self.set_step(step)
        self.losses = torch.zeros(L, dtype=torch.float32, device=self.dev)

    def device_tokens(self, tokens: np.ndarray):
        t = self.torch.from_numpy(np.ascontiguousarray(tokens, dtype=np.int32)).to(self.dev)
        self.torch.cuda.synchronize(self.dev)
        return t

    def step(self, tokens, schedule="overlap", losses=None, wait_current=True):
        if wait_current:
            self.sf.wait_stream(self.torch.cuda.current_stream(self.dev))
        sched = SCHEDULES[schedule] if isinstance(schedule, str) else int(schedule)
        out = self.losses if losses is None else losses
        _check(lib().erase_tf_step(self.ctx, c_void_p(tokens.data_ptr()), sched, c_void_p(out.data_ptr())),
               "erase_tf_step", self.ctx)
        return out

    def sync(self):
        _check(lib().erase_tf_sync(self.ctx), "erase_tf_sync", self.ctx)

    def get_step(self) -> int:
        t = c_int64(0)
        _check(lib().erase_tf_get_step(self.ctx, ctypes.byref(t)), "erase_tf_get_step", self.ctx)
        return t.value

    def set_step(self, t: int):
        _check(lib().erase_tf_set_step(self.ctx, int(t)), "erase_tf_set_step", self.ctx)

    def refresh_weights(self):
        _check(lib().erase_tf_refresh_weights(self.ctx), "erase_tf_refresh_weights", self.ctx)

    def set_timing(self, on: bool):
        _check(lib().erase_tf_set_timing(self.ctx, 1 if on else 0), "erase_tf_set_timing", self.ctx)

    def read_timing(self):
        n = c_int32(0)
        cap = 8192
        arr = (KernelTime * cap)()
        _check(lib().erase_tf_read_timing(self.ctx, arr, cap, ctypes.byref(n)), "erase_tf_read_timing", self.ctx)
        return [dict(kind=TF_KERNEL_KINDS[a.kind], block=a.block, layer=a.layer, stream=a.stream,
                     start_ms=a.start_ms, end_ms=a.end_ms, tile_m=a.tile_m, tile_n=a.tile_n, split=a.split,
                     grid=a.grid, flops=a.flops, bytes=a.bytes)
                for a in arr[:min(n.value, cap)]]

    def tensor(self, block: int, name: str, rows: int, cols: int, dtype="bf16"):
        """Copy of a stored tensor ([rows][cols] of its pitch) as float32 numpy."""
        torch = self.torch
        p, ld = c_void_p(), c_int64(0)
        _check(lib().erase_tf_tensor(self.ctx, block, TENSORS[name], ctypes.byref(p), ctypes.byref(ld)),
               "erase_tf_tensor", self.ctx)
        esz = 2 if dtype == "bf16" else 4
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.sync()
        # wrap the device range through a raw byte view of the workspace
        off = p.value - self.ws.data_ptr()
        assert 0 <= off and off + rows * ld.value * esz <= self.ws.numel()
        raw = self.ws[off:off + rows * ld.value * esz].view(tdt).view(rows, ld.value)
        return raw[:, :cols].float().cpu().numpy()

    def flat_state(self):
        self.sync()
        return ([t.detach().cpu().numpy().copy() for t in self.param],
                [t.detach().cpu().numpy().copy() for t in self.m],
                [t.detach().cpu().numpy().copy() for t in self.v],
                [None if t is None else t.detach().cpu().numpy().copy() for t in self.grad])

    def close(self):
        if getattr(self, "ctx", None):
            lib().erase_tf_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
