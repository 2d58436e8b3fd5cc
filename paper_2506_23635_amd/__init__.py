"""Python binding of the gfx950 MoE library (libmoe.so, C-ABI in include/moe.h).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  PyTorch is used for device memory and streams; if the library is not
built this module raises on first use instead of falling back to anything.

The functions carry the C names (moe_init, moe_route, moe_forward, ...).
``MoeLayer`` bundles the caller-owned arena and workspace with a context.
"""
from __future__ import annotations

import ctypes
import os

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libmoe.so")

MOE_OK = 0
MOE_PARTIAL_F32 = 0x1   # moe_config.flags: y of moe_forward is fp32 [T, d]
DIAG_MAX_WG = 512    # MOE_DIAG_MAX_WG of include/moe.h
WS_REGIONS = ["route_partials", "logits", "topk_idx", "topk_w", "counts", "offsets", "pair_row",
              "row_token", "active", "tiles", "n_tiles", "h", "o"]   # moe_ws_region order
STATUS_NAMES = {0: "MOE_OK", -1: "MOE_E_ARG", -2: "MOE_E_SHAPE", -3: "MOE_E_ALIGN",
                -4: "MOE_E_CAPACITY", -5: "MOE_E_STATE", -6: "MOE_E_HIP"}

EXPORTED = ["moe_weight_bytes", "moe_workspace_bytes", "moe_workspace_map", "moe_init",
            "moe_load_expert",
            "moe_load_router", "moe_route", "moe_forward", "moe_forward_static",
            "moe_forward_stack", "moe_forward_layers", "moe_forward_residual",
            "moe_intermediates", "moe_profile_enable", "moe_profile_read",
            "moe_profile_gemm_timeline", "moe_destroy",
            "moe_last_error", "moe_status_string", "moe_diag_stream_read", "moe_diag_bf16",
            # include/attn.h
            "attn_weight_bytes", "attn_cache_bytes", "attn_workspace_bytes", "attn_init",
            "attn_load_layer", "attn_load_post_norm", "attn_forward", "attn_forward_norm",
            "attn_intermediates", "attn_profile_enable", "attn_profile_read", "attn_destroy",
            "attn_last_error"]

ATTN_KERNEL_KINDS = ["norm", "qkv", "score", "combine", "out", "pack", "rope", "residual",
                     "post_norm"]

KERNEL_KINDS = ["router", "route", "decode_gateup", "decode_down", "gemm_gateup", "gemm_down",
                "combine", "pack"]


class MoeConfig(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("expert_begin", ctypes.c_int32), ("n_local_experts", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("max_tokens", ctypes.c_int32),
                ("flags", ctypes.c_int32)]


class MoeRouting(ctypes.Structure):
    _fields_ = [("logits", ctypes.c_void_p), ("topk_idx", ctypes.c_void_p),
                ("topk_w", ctypes.c_void_p), ("counts", ctypes.c_void_p),
                ("offsets", ctypes.c_void_p), ("pair_row", ctypes.c_void_p),
                ("row_token", ctypes.c_void_p), ("T", ctypes.c_int32),
                ("layer", ctypes.c_int32)]


class AttnConfig(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("max_seq", ctypes.c_int32),
                ("max_tokens", ctypes.c_int32), ("rope_theta", ctypes.c_float),
                ("norm_eps", ctypes.c_float), ("flags", ctypes.c_int32)]


class MoeError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def lib():
    """The loaded libmoe.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        # torch first: its HIP runtime then also serves this library (one
        # runtime per process, so torch streams are valid handles here)
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        P, I = ctypes.c_void_p, ctypes.c_int32
        cfgp = ctypes.POINTER(MoeConfig)
        L.moe_weight_bytes.argtypes = [cfgp]
        L.moe_weight_bytes.restype = ctypes.c_size_t
        L.moe_workspace_bytes.argtypes = [cfgp]
        L.moe_workspace_bytes.restype = ctypes.c_size_t
        L.moe_workspace_map.argtypes = [cfgp, P, P, I]
        L.moe_workspace_map.restype = ctypes.c_int32
        L.moe_init.argtypes = [cfgp, P, P, ctypes.POINTER(P)]
        L.moe_load_expert.argtypes = [P, I, I, P, P, P, I, P]
        L.moe_load_router.argtypes = [P, I, P, P, I, P]
        L.moe_route.argtypes = [P, I, P, I, P, ctypes.POINTER(MoeRouting), P]
        L.moe_forward.argtypes = [P, I, P, I, ctypes.POINTER(MoeRouting), P, P]
        L.moe_forward_static.argtypes = [P, I, P, I, P, P]
        L.moe_forward_stack.argtypes = [P, P, I, P]
        L.moe_forward_layers.argtypes = [P, I, I, P, I, P]
        L.moe_forward_residual.argtypes = [P, I, P, P, I, P]
        L.moe_intermediates.argtypes = [P, ctypes.POINTER(P), ctypes.POINTER(P)]
        L.moe_profile_enable.argtypes = [P, I]
        L.moe_profile_read.argtypes = [P, P, P, P]
        L.moe_profile_gemm_timeline.argtypes = [P, P, P, I]
        L.moe_destroy.argtypes = [P]
        L.moe_destroy.restype = None
        L.moe_last_error.argtypes = [P]
        L.moe_last_error.restype = ctypes.c_char_p
        L.moe_status_string.argtypes = [ctypes.c_int]
        L.moe_status_string.restype = ctypes.c_char_p
        L.moe_diag_stream_read.argtypes = [P, ctypes.c_uint64, P, P]
        L.moe_diag_bf16.argtypes = [P, P, ctypes.c_uint64, P]
        acfg = ctypes.POINTER(AttnConfig)
        for fn in ("attn_weight_bytes", "attn_cache_bytes", "attn_workspace_bytes"):
            getattr(L, fn).argtypes = [acfg]
            getattr(L, fn).restype = ctypes.c_size_t
        L.attn_init.argtypes = [acfg, P, P, P, ctypes.POINTER(P)]
        L.attn_load_layer.argtypes = [P, I, P, P, P, I, P]
        L.attn_forward.argtypes = [P, I, P, P, I, I, P]
        L.attn_load_post_norm.argtypes = [P, I, P, I, P]
        L.attn_forward_norm.argtypes = [P, I, P, P, P, I, I, P]
        L.attn_intermediates.argtypes = [P] + [ctypes.POINTER(P)] * 5
        L.attn_profile_enable.argtypes = [P, I]
        L.attn_profile_read.argtypes = [P, P, P, P]
        L.attn_destroy.argtypes = [P]
        L.attn_destroy.restype = None
        L.attn_last_error.argtypes = [P]
        L.attn_last_error.restype = ctypes.c_char_p
        for fn in ("attn_init", "attn_load_layer", "attn_load_post_norm", "attn_forward",
                   "attn_forward_norm", "attn_intermediates",
                   "attn_profile_enable", "attn_profile_read"):
            getattr(L, fn).restype = ctypes.c_int
        for fn in ("moe_init", "moe_load_expert", "moe_load_router", "moe_route", "moe_forward",
                   "moe_forward_static", "moe_forward_stack", "moe_forward_layers",
                   "moe_forward_residual",
                   "moe_intermediates", "moe_profile_enable",
                   "moe_profile_read", "moe_profile_gemm_timeline", "moe_diag_stream_read",
                   "moe_diag_bf16"):
            getattr(L, fn).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(ctx, status: int):
    if status != MOE_OK:
        msg = lib().moe_last_error(ctx).decode()
        raise MoeError(status, msg)


def make_config(d_model, ffn_dim, n_experts, top_k, expert_begin=0, n_local_experts=0,
                n_layers=1, max_tokens=1, flags=0) -> MoeConfig:
    return MoeConfig(d_model, ffn_dim, n_experts, top_k, expert_begin,
                     n_local_experts or n_experts, n_layers, max_tokens, flags)


def moe_weight_bytes(cfg: MoeConfig) -> int:
    return int(lib().moe_weight_bytes(ctypes.byref(cfg)))


def moe_workspace_bytes(cfg: MoeConfig) -> int:
    return int(lib().moe_workspace_bytes(ctypes.byref(cfg)))


def moe_workspace_map(cfg: MoeConfig) -> dict:
    """{region name: (byte offset, bytes)} of the workspace for cfg."""
    n = len(WS_REGIONS)
    off = (ctypes.c_uint64 * n)()
    nb = (ctypes.c_uint64 * n)()
    got = lib().moe_workspace_map(ctypes.byref(cfg), off, nb, n)
    if got != n:
        raise MoeError(-2, "invalid config" if got == 0 else f"{got} regions, expected {n}")
    return {name: (int(off[i]), int(nb[i])) for i, name in enumerate(WS_REGIONS)}


def moe_init(cfg: MoeConfig, arena_ptr: int, workspace_ptr: int) -> int:
    out = ctypes.c_void_p()
    _check(None, lib().moe_init(ctypes.byref(cfg), arena_ptr, workspace_ptr, ctypes.byref(out)))
    return out.value


def moe_load_expert(ctx, layer, expert, gate_ptr, up_ptr, down_ptr, src_on_device, stream=0):
    _check(ctx, lib().moe_load_expert(ctx, layer, expert, gate_ptr, up_ptr, down_ptr,
                                      src_on_device, stream))


def moe_load_router(ctx, layer, wr_ptr, bias_ptr, src_on_device, stream=0):
    _check(ctx, lib().moe_load_router(ctx, layer, wr_ptr, bias_ptr, src_on_device, stream))


def moe_route(ctx, layer, x_ptr, T, logits_in_ptr=None, stream=0) -> MoeRouting:
    r = MoeRouting()
    _check(ctx, lib().moe_route(ctx, layer, x_ptr, T, logits_in_ptr, ctypes.byref(r), stream))
    return r


def moe_forward(ctx, layer, x_ptr, T, routing, y_ptr, stream=0):
    rp = ctypes.byref(routing) if routing is not None else None
    _check(ctx, lib().moe_forward(ctx, layer, x_ptr, T, rp, y_ptr, stream))


def moe_forward_static(ctx, layer, x_ptr, T, y_ptr, stream=0):
    _check(ctx, lib().moe_forward_static(ctx, layer, x_ptr, T, y_ptr, stream))


def moe_forward_stack(ctx, x_ptr, T, stream=0):
    _check(ctx, lib().moe_forward_stack(ctx, x_ptr, T, stream))


def moe_forward_layers(ctx, first, n, x_ptr, T, stream=0):
    _check(ctx, lib().moe_forward_layers(ctx, first, n, x_ptr, T, stream))


def moe_forward_residual(ctx, layer, x_ptr, r_ptr, T, stream=0):
    _check(ctx, lib().moe_forward_residual(ctx, layer, x_ptr, r_ptr, T, stream))


def moe_diag_stream_read(src_ptr, nbytes, out_ptr, stream=0):
    """One plain streaming read of nbytes at src_ptr; workgroup b writes the
    XOR of its words to the 4 uint32 at out_ptr + 16 b (device pointers; out
    holds DIAG_MAX_WG x 4 uint32, zeroed by the caller; see include/moe.h)."""
    st = lib().moe_diag_stream_read(src_ptr, nbytes, out_ptr, stream)
    if st != MOE_OK:
        raise MoeError(st, lib().moe_status_string(st).decode())


def moe_diag_bf16(src_ptr, dst_ptr, n, stream=0):
    """dst[i] = bf16(src[i]), i < n, by the gate/up epilogue's hardware
    conversion (device pointers; see include/moe.h)."""
    st = lib().moe_diag_bf16(src_ptr, dst_ptr, n, stream)
    if st != MOE_OK:
        raise MoeError(st, lib().moe_status_string(st).decode())


def moe_intermediates(ctx):
    h = ctypes.c_void_p()
    o = ctypes.c_void_p()
    _check(ctx, lib().moe_intermediates(ctx, ctypes.byref(h), ctypes.byref(o)))
    return h.value, o.value


def moe_profile_enable(ctx, max_launches: int):
    _check(ctx, lib().moe_profile_enable(ctx, max_launches))


def moe_profile_read(ctx):
    """{kind: (total_ms, launches)} since the last read, and the dropped count."""
    n = len(KERNEL_KINDS)
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int64 * n)()
    dropped = ctypes.c_int64()
    _check(ctx, lib().moe_profile_read(ctx, ms, cnt, ctypes.byref(dropped)))
    return {k: (ms[i], cnt[i]) for i, k in enumerate(KERNEL_KINDS)}, dropped.value


def moe_profile_gemm_timeline(ctx, gateup_ptr, down_ptr, max_wg: int):
    """Per-workgroup GEMM timelines into two uint64 [max_wg][8] device
    buffers (0 / None turns it off); see include/moe.h for the fields."""
    _check(ctx, lib().moe_profile_gemm_timeline(ctx, gateup_ptr, down_ptr, max_wg))


def moe_destroy(ctx):
    if ctx:
        lib().moe_destroy(ctx)


def moe_last_error(ctx) -> str:
    return lib().moe_last_error(ctx).decode()


# ------------------------------------------------------------ torch helper --

def _tensor_ptr(t, name, min_numel, dtypes, device):
    """Checks a torch tensor before its address crosses the C-ABI, which
    cannot see sizes: one of `dtypes`, contiguous, on `device` (None: any),
    at least `min_numel` elements.  Returns its data pointer."""
    if t is None:
        raise MoeError(-1, f"{name} is None")
    if t.dtype not in dtypes:
        raise MoeError(-1, f"{name} has dtype {t.dtype}, expected one of {list(dtypes)}")
    if not t.is_contiguous():
        raise MoeError(-1, f"{name} must be contiguous")
    if device is not None and t.device != device:
        raise MoeError(-1, f"{name} is on {t.device}, expected {device}")
    if t.numel() < min_numel:
        raise MoeError(-2, f"{name} has {t.numel()} elements, the call uses {min_numel}")
    return t.data_ptr()


def _bf16_types(torch):
    # bf16 tensors may arrive as bfloat16 or as their 16-bit integer bits
    return (torch.bfloat16, torch.int16, torch.uint16)

class MoeLayer:
    """Owns a context plus its torch-allocated arena and workspace on one GPU.

    Only allocation and pointer marshalling happen here; all compute is in
    the library."""

    def __init__(self, cfg: MoeConfig, device="cuda", arena=None, workspace=None):
        """arena / workspace: caller-owned uint8 device tensors of at least
        moe_weight_bytes / moe_workspace_bytes (allocated here if None)."""
        import torch
        self.torch = torch
        self.cfg = cfg
        self.device = torch.device(device)
        if self.device.type != "cuda":
            raise MoeError(-1, f"the layer runs on a GPU, not on {self.device}")
        if self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        wb = moe_weight_bytes(cfg)
        sb = moe_workspace_bytes(cfg)
        if wb == 0 or sb == 0:
            raise MoeError(-2, "invalid config")
        if arena is not None and arena.numel() < wb or workspace is not None and workspace.numel() < sb:
            raise MoeError(-1, "arena or workspace smaller than the config needs")
        self.arena = torch.empty(wb, dtype=torch.uint8, device=self.device) if arena is None else arena
        self.workspace = (torch.empty(sb, dtype=torch.uint8, device=self.device)
                          if workspace is None else workspace)
        self.ctx = moe_init(cfg, _tensor_ptr(self.arena, "arena", wb, (torch.uint8,), self.device),
                            _tensor_ptr(self.workspace, "workspace", sb, (torch.uint8,), self.device))

    @property
    def stream(self) -> int:
        return self.torch.cuda.current_stream(self.device).cuda_stream

    def close(self):
        if getattr(self, "ctx", None):
            moe_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # Tensors: row-major, contiguous; bf16 as bfloat16 or int16/uint16 bits;
    # activations on self.device, weights on self.device or all on the host.
    # Every tensor is checked (dtype, layout, device, element count) before
    # its address is handed to the library.
    def _src_device(self, *ts):
        on_dev = ts[0].is_cuda
        if any(t is not None and t.is_cuda != on_dev for t in ts):
            raise MoeError(-1, "weights must be all on the GPU or all on the host")
        return on_dev, (self.device if on_dev else self.torch.device("cpu"))

    def load_expert(self, layer, expert, gate, up, down):
        c, bf = self.cfg, _bf16_types(self.torch)
        on_dev, dev = self._src_device(gate, up, down)
        n = c.d_model * c.ffn_dim
        moe_load_expert(self.ctx, layer, expert, _tensor_ptr(gate, "gate", n, bf, dev),
                        _tensor_ptr(up, "up", n, bf, dev), _tensor_ptr(down, "down", n, bf, dev),
                        int(on_dev), self.stream if on_dev else 0)

    def load_router(self, layer, wr, bias=None):
        c, f32 = self.cfg, (self.torch.float32,)
        on_dev, dev = self._src_device(wr, bias)
        moe_load_router(self.ctx, layer, _tensor_ptr(wr, "wr", c.d_model * c.n_experts, f32, dev),
                        _tensor_ptr(bias, "bias", c.n_experts, f32, dev) if bias is not None else None,
                        int(on_dev), self.stream if on_dev else 0)

    def _tokens(self, x, T):
        T = x.shape[0] if T is None else int(T)
        if T < 0:
            raise MoeError(-1, "T is negative")
        return T

    def route(self, layer, x, T=None, logits_in=None) -> MoeRouting:
        if x is None and logits_in is None:
            raise MoeError(-1, "route needs x or logits_in")
        T = self._tokens(x if x is not None else logits_in, T)
        d, E = self.cfg.d_model, self.cfg.n_experts
        xp = _tensor_ptr(x, "x", T * d, _bf16_types(self.torch), self.device) if x is not None else None
        lp = (_tensor_ptr(logits_in, "logits_in", T * E, (self.torch.float32,), self.device)
              if logits_in is not None else None)
        return moe_route(self.ctx, layer, xp, T, lp, self.stream)

    def forward(self, layer, x, y, routing=None, T=None):
        """y: bf16 [T, d], or fp32 [T, d] when the config has MOE_PARTIAL_F32."""
        T = self._tokens(x, T)
        n, bf = T * self.cfg.d_model, _bf16_types(self.torch)
        ytypes = (self.torch.float32,) if self.cfg.flags & MOE_PARTIAL_F32 else bf
        moe_forward(self.ctx, layer, _tensor_ptr(x, "x", n, bf, self.device), T, routing,
                    _tensor_ptr(y, "y", n, ytypes, self.device), self.stream)

    def forward_static(self, layer, x, y, T=None):
        """moe_forward_static: the layer with internal routing on the
        library's static device scratch (no workspace use, no allocation)."""
        T = self._tokens(x, T)
        n, bf = T * self.cfg.d_model, _bf16_types(self.torch)
        ytypes = (self.torch.float32,) if self.cfg.flags & MOE_PARTIAL_F32 else bf
        moe_forward_static(self.ctx, layer, _tensor_ptr(x, "x", n, bf, self.device), T,
                           _tensor_ptr(y, "y", n, ytypes, self.device), self.stream)

    def forward_stack(self, x, T=None):
        T = self._tokens(x, T)
        moe_forward_stack(self.ctx, _tensor_ptr(x, "x", T * self.cfg.d_model, _bf16_types(self.torch),
                                                self.device), T, self.stream)

    def forward_residual(self, layer, x, r, T=None):
        """moe_forward_residual: r = bf16(r + bf16(layer(x))) in place."""
        T = self._tokens(x, T)
        n, bf = T * self.cfg.d_model, _bf16_types(self.torch)
        moe_forward_residual(self.ctx, layer, _tensor_ptr(x, "x", n, bf, self.device),
                             _tensor_ptr(r, "r", n, bf, self.device), T, self.stream)

    def forward_layers(self, first, n, x, T=None):
        """moe_forward_layers: layers first .. first+n-1, x = bf16(x + y) in place."""
        T = self._tokens(x, T)
        moe_forward_layers(self.ctx, first, n,
                           _tensor_ptr(x, "x", T * self.cfg.d_model, _bf16_types(self.torch),
                                       self.device), T, self.stream)

    def routing_tensors(self, r: MoeRouting):
        """Copies the routing views (device) to host numpy arrays."""
        import numpy as np
        torch = self.torch
        T, E, k = r.T, self.cfg.n_experts, self.cfg.top_k

        def dev(ptr, n, dtype):
            buf = torch.empty(n, dtype=dtype, device=self.device)
            if n:
                _copy_dev(buf.data_ptr(), ptr, buf.numel() * buf.element_size())
            return buf

        torch.cuda.synchronize(self.device)
        out = {
            "logits": dev(r.logits, T * E, torch.float32).cpu().numpy().reshape(T, E),
            "idx": dev(r.topk_idx, T * k, torch.int32).cpu().numpy().reshape(T, k),
            "w": dev(r.topk_w, T * k, torch.float32).cpu().numpy().reshape(T, k),
            "counts": dev(r.counts, E, torch.int32).cpu().numpy(),
            "offsets": dev(r.offsets, E + 1, torch.int32).cpu().numpy(),
            "pair_row": dev(r.pair_row, T * k, torch.int32).cpu().numpy().reshape(T, k),
        }
        n_rows = int(out["offsets"][-1])
        out["row_token"] = dev(r.row_token, n_rows, torch.int32).cpu().numpy()
        assert out["logits"].dtype == np.float32
        return out


_hip = None
HIP_ATTR_WALL_CLOCK_RATE = 10019   # hipDeviceAttributeWallClockRate (kHz)


def _hip_runtime():
    """The HIP runtime already mapped into this process (torch's)."""
    global _hip
    if _hip is None:
        lib()
        path = "libamdhip64.so"
        with open(f"/proc/{os.getpid()}/maps") as fh:
            for ln in fh:
                if "libamdhip64" in ln and ln.split()[-1].startswith("/"):
                    path = ln.split()[-1]
                    break
        h = ctypes.CDLL(path)
        h.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        h.hipMemcpy.restype = ctypes.c_int
        h.hipDeviceGetAttribute.argtypes = [ctypes.POINTER(ctypes.c_int), ctypes.c_int, ctypes.c_int]
        h.hipDeviceGetAttribute.restype = ctypes.c_int
        _hip = h
    return _hip


def _copy_dev(dst_ptr: int, src_ptr: int, nbytes: int):
    """Device-to-device copy through the HIP runtime (read-back helper)."""
    rc = _hip_runtime().hipMemcpy(ctypes.c_void_p(dst_ptr), ctypes.c_void_p(src_ptr), nbytes, 3)
    if rc != 0:
        raise RuntimeError(f"hipMemcpy failed: {rc}")


def wall_clock_hz(device: int = 0) -> float:
    """Rate of the constant counter the GEMM timeline's [0], [1] fields read
    (hipDeviceAttributeWallClockRate)."""
    v = ctypes.c_int()
    rc = _hip_runtime().hipDeviceGetAttribute(ctypes.byref(v), HIP_ATTR_WALL_CLOCK_RATE, device)
    if rc != 0:
        raise RuntimeError(f"hipDeviceGetAttribute failed: {rc}")
    return v.value * 1e3


# ------------------------------------------------------- attention block --

def _acheck(ctx, status: int):
    if status != MOE_OK:
        raise MoeError(status, lib().attn_last_error(ctx).decode())


def make_attn_config(d_model, n_heads, n_kv_heads, head_dim, n_layers=1, max_seq=4096,
                     max_tokens=16, rope_theta=5e5, norm_eps=1e-5, flags=0) -> AttnConfig:
    return AttnConfig(d_model, n_heads, n_kv_heads, head_dim, n_layers, max_seq, max_tokens,
                      rope_theta, norm_eps, flags)


def attn_weight_bytes(cfg: AttnConfig) -> int:
    return int(lib().attn_weight_bytes(ctypes.byref(cfg)))


def attn_cache_bytes(cfg: AttnConfig) -> int:
    return int(lib().attn_cache_bytes(ctypes.byref(cfg)))


def attn_workspace_bytes(cfg: AttnConfig) -> int:
    return int(lib().attn_workspace_bytes(ctypes.byref(cfg)))


def attn_init(cfg: AttnConfig, arena_ptr: int, cache_ptr: int, workspace_ptr: int) -> int:
    out = ctypes.c_void_p()
    _acheck(None, lib().attn_init(ctypes.byref(cfg), arena_ptr, cache_ptr, workspace_ptr,
                                  ctypes.byref(out)))
    return out.value


def attn_load_layer(ctx, layer, gamma_ptr, wqkv_ptr, wo_ptr, src_on_device, stream=0):
    _acheck(ctx, lib().attn_load_layer(ctx, layer, gamma_ptr, wqkv_ptr, wo_ptr, src_on_device,
                                       stream))


def attn_forward(ctx, layer, x_ptr, y_ptr, T, pos0, stream=0):
    _acheck(ctx, lib().attn_forward(ctx, layer, x_ptr, y_ptr, T, pos0, stream))


def attn_load_post_norm(ctx, layer, gamma2_ptr, src_on_device, stream=0):
    _acheck(ctx, lib().attn_load_post_norm(ctx, layer, gamma2_ptr, src_on_device, stream))


def attn_forward_norm(ctx, layer, x_ptr, y_ptr, z_ptr, T, pos0, stream=0):
    _acheck(ctx, lib().attn_forward_norm(ctx, layer, x_ptr, y_ptr, z_ptr, T, pos0, stream))


def attn_intermediates(ctx):
    ptrs = [ctypes.c_void_p() for _ in range(5)]
    _acheck(ctx, lib().attn_intermediates(ctx, *[ctypes.byref(p) for p in ptrs]))
    return [p.value for p in ptrs]


def attn_profile_enable(ctx, max_launches: int):
    _acheck(ctx, lib().attn_profile_enable(ctx, max_launches))


def attn_profile_read(ctx):
    n = len(ATTN_KERNEL_KINDS)
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int64 * n)()
    dropped = ctypes.c_int64()
    _acheck(ctx, lib().attn_profile_read(ctx, ms, cnt, ctypes.byref(dropped)))
    return {k: (ms[i], cnt[i]) for i, k in enumerate(ATTN_KERNEL_KINDS)}, dropped.value


class AttnLayer:
    """Owns an attention context plus its torch-allocated weight arena, key/value
    cache and workspace on one GPU (argument marshalling only)."""

    def __init__(self, cfg: AttnConfig, device="cuda", arena=None, cache=None, workspace=None):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.device = torch.device(device)
        if self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        wb, cb, sb = attn_weight_bytes(cfg), attn_cache_bytes(cfg), attn_workspace_bytes(cfg)
        if not (wb and cb and sb):
            raise MoeError(-2, "invalid attention config")

        def buf(t, n, name):
            if t is None:
                return torch.empty(n, dtype=torch.uint8, device=self.device)
            _tensor_ptr(t, name, n, (torch.uint8,), self.device)
            return t
        self.arena = buf(arena, wb, "arena")
        self.cache = buf(cache, cb, "cache")
        self.workspace = buf(workspace, sb, "workspace")
        self.ctx = attn_init(cfg, self.arena.data_ptr(), self.cache.data_ptr(),
                             self.workspace.data_ptr())

    @property
    def stream(self) -> int:
        return self.torch.cuda.current_stream(self.device).cuda_stream

    def close(self):
        if getattr(self, "ctx", None):
            lib().attn_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def cache_views(self, layer):
        """(K, V) of a layer as bf16-bit int16 views [n_kv_heads, max_seq, head_dim]."""
        c = self.cfg
        per = c.n_kv_heads * c.max_seq * c.head_dim
        allc = self.cache.view(self.torch.int16).view(c.n_layers, 2, per)
        shape = (c.n_kv_heads, c.max_seq, c.head_dim)
        return allc[layer, 0].view(shape), allc[layer, 1].view(shape)

    def load_layer(self, layer, gamma, wqkv, wo):
        c, bf = self.cfg, _bf16_types(self.torch)
        on_dev = wqkv.is_cuda
        if gamma.is_cuda != on_dev or wo.is_cuda != on_dev:
            raise MoeError(-1, "weights must be all on the GPU or all on the host")
        dev = self.device if on_dev else self.torch.device("cpu")
        nq = c.n_heads * c.head_dim
        nqkv = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim
        attn_load_layer(self.ctx, layer,
                        _tensor_ptr(gamma, "gamma", c.d_model, (self.torch.float32,), dev),
                        _tensor_ptr(wqkv, "wqkv", c.d_model * nqkv, bf, dev),
                        _tensor_ptr(wo, "wo", nq * c.d_model, bf, dev), int(on_dev),
                        self.stream if on_dev else 0)

    def forward(self, layer, x, y, pos0, T=None):
        T = x.shape[0] if T is None else int(T)
        n, bf = T * self.cfg.d_model, _bf16_types(self.torch)
        attn_forward(self.ctx, layer, _tensor_ptr(x, "x", n, bf, self.device),
                     _tensor_ptr(y, "y", n, bf, self.device), T, pos0, self.stream)

    def load_post_norm(self, layer, gamma2):
        on_dev = gamma2.is_cuda
        dev = self.device if on_dev else self.torch.device("cpu")
        attn_load_post_norm(self.ctx, layer,
                            _tensor_ptr(gamma2, "gamma2", self.cfg.d_model, (self.torch.float32,), dev),
                            int(on_dev), self.stream if on_dev else 0)

    def forward_norm(self, layer, x, y, z, pos0, T=None):
        """attn_forward_norm: y = x + attention, z = the post-attention norm of y."""
        T = x.shape[0] if T is None else int(T)
        n, bf = T * self.cfg.d_model, _bf16_types(self.torch)
        attn_forward_norm(self.ctx, layer, _tensor_ptr(x, "x", n, bf, self.device),
                          _tensor_ptr(y, "y", n, bf, self.device),
                          _tensor_ptr(z, "z", n, bf, self.device), T, pos0, self.stream)

    def intermediates(self, T):
        """Copies of the last forward's h, qkv, q, a, o (numpy; bf16 as uint16)."""
        import numpy as np
        torch = self.torch
        c = self.cfg
        nq = c.n_heads * c.head_dim
        nqkv = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim
        ptrs = attn_intermediates(self.ctx)
        spec = [(c.d_model, torch.int16), (nqkv, torch.float32), (nq, torch.int16),
                (nq, torch.int16), (c.d_model, torch.float32)]
        out = []
        torch.cuda.synchronize(self.device)
        for ptr, (w, dt) in zip(ptrs, spec):
            t = torch.empty((T, w), dtype=dt, device=self.device)
            _copy_dev(t.data_ptr(), ptr, t.numel() * t.element_size())
            a = t.cpu().numpy()
            out.append(a.view(np.uint16) if dt == torch.int16 else a)
        return dict(zip(["h", "qkv", "q", "a", "o"], out))
