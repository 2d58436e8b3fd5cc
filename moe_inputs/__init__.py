"""Seeded synthetic inputs for the DBRX-shaped MoE layer.

This module is shared by the tests, the benchmark and the oracle's callers.
It holds no arithmetic of the layer itself: it only turns (seed, stream,
element index) into tensor bits (definition in ``philox_gen.h``) and records
the workload recipes (shapes, value scales, routing skew) that stand in for
the paper's DBRX Instruct workload (Sec. 5.1, Table tab:vars: D_embed 6144,
D_ffn 10752, 16 experts, top-4, bf16).

Both a host build (gcc, OpenMP) and a device build (hipcc, writes straight
into HBM) exist; they produce identical bits.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_HOST_LIB = os.path.join(HERE, "libmoe_inputs_host.so")
_DEV_LIB = os.path.join(HERE, "libmoe_inputs_device.so")

# Stream kinds: stream id = kind | expert << 4 | layer << 12.
KIND_X = 1
KIND_ROUTER = 2
KIND_BIAS = 3
KIND_GATE = 4
KIND_UP = 5
KIND_DOWN = 6
# attention block inputs
KIND_ATTN_X = 7
KIND_GAMMA = 8
KIND_WQKV = 9
KIND_WO = 10
KIND_KCACHE = 11
KIND_VCACHE = 12

# sd of z = 2*S - 8*65535 where S is a sum of eight uniform 16-bit integers
_SD_Z = 2.0 * math.sqrt(8.0 * (65536.0 ** 2 - 1.0) / 12.0)


def scale_for(sigma: float) -> float:
    """The double c with value = z * c having standard deviation sigma."""
    return float(sigma) / _SD_Z


def stream_id(kind: int, layer: int = 0, expert: int = 0) -> int:
    if not (0 < kind < 16 and 0 <= expert < 256 and 0 <= layer < (1 << 20)):
        raise ValueError("stream id out of range")
    return kind | (expert << 4) | (layer << 12)


def build(force: bool = True) -> None:
    """Compile the host (gcc) and device (hipcc, gfx950) generator libraries."""
    src_h = os.path.join(HERE, "philox_gen.h")
    src_c = os.path.join(HERE, "gen_host.c")
    src_d = os.path.join(HERE, "gen_device.hip")

    def stale(lib, srcs):
        return force or not os.path.exists(lib) or any(
            os.path.getmtime(s) > os.path.getmtime(lib) for s in srcs)

    if stale(_HOST_LIB, [src_h, src_c]):
        tmp = _HOST_LIB + ".tmp"
        subprocess.run(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC",
                        "-shared", "-Wall", "-o", tmp, src_c], check=True)
        os.replace(tmp, _HOST_LIB)
    if stale(_DEV_LIB, [src_h, src_d]):
        tmp = _DEV_LIB + ".tmp"
        subprocess.run(["hipcc", "--offload-arch=gfx950", "-O3", "-ffp-contract=off", "-fPIC",
                        "-shared", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                        "-o", tmp, src_d], check=True, stderr=subprocess.DEVNULL)
        os.replace(tmp, _DEV_LIB)


_host = None
_dev = None


def _host_lib():
    global _host
    if _host is None:
        if not os.path.exists(_HOST_LIB):
            build(force=False)
        lib = ctypes.CDLL(_HOST_LIB)
        lib.moe_gen_fill_bf16.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64,
                                          ctypes.c_int64, ctypes.c_double, ctypes.c_void_p]
        lib.moe_gen_fill_f32.argtypes = lib.moe_gen_fill_bf16.argtypes
        lib.moe_gen_philox.argtypes = [ctypes.c_void_p] * 3
        lib.moe_gen_z_at.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64]
        lib.moe_gen_z_at.restype = ctypes.c_int32
        lib.moe_gen_bf16_rne_host.argtypes = [ctypes.c_double]
        lib.moe_gen_bf16_rne_host.restype = ctypes.c_uint16
        _host = lib
    return _host


def _dev_lib():
    global _dev
    if _dev is None:
        if not os.path.exists(_DEV_LIB):
            raise RuntimeError(f"device input generator not built: {_DEV_LIB}")
        import torch  # noqa: F401  (load torch's HIP runtime first: one runtime per process)
        lib = ctypes.CDLL(_DEV_LIB)
        for fn in (lib.moe_gen_fill_bf16_device, lib.moe_gen_fill_f32_device):
            fn.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int64,
                           ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p]
            fn.restype = ctypes.c_int
        _dev = lib
    return _dev


def philox4x32_10(counter, key):
    lib = _host_lib()
    c = (ctypes.c_uint32 * 4)(*counter)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    lib.moe_gen_philox(c, k, o)
    return [int(v) for v in o]


def z_at(seed: int, stream: int, index: int) -> int:
    return int(_host_lib().moe_gen_z_at(seed, stream, index))


def bf16_rne(v: float) -> int:
    """The generator's own double->bf16 rounding (used only to build inputs)."""
    return int(_host_lib().moe_gen_bf16_rne_host(float(v)))


def gen_bf16(seed: int, stream: int, shape, sigma: float, start: int = 0) -> np.ndarray:
    """bf16 tensor as uint16 bit patterns, row-major, elements start.. of the stream."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    _host_lib().moe_gen_fill_bf16(seed, stream, start, n, scale_for(sigma),
                                  out.ctypes.data)
    return out.reshape(shape)


def gen_f32(seed: int, stream: int, shape, sigma: float, start: int = 0) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    _host_lib().moe_gen_fill_f32(seed, stream, start, n, scale_for(sigma), out.ctypes.data)
    return out.reshape(shape)


def gen_bf16_device(seed: int, stream: int, n: int, sigma: float, dst_ptr: int,
                    hip_stream: int = 0, start: int = 0) -> None:
    rc = _dev_lib().moe_gen_fill_bf16_device(seed, stream, start, n, scale_for(sigma),
                                             ctypes.c_void_p(dst_ptr),
                                             ctypes.c_void_p(hip_stream))
    if rc != 0:
        raise RuntimeError(f"moe_gen_fill_bf16_device failed: {rc}")


def gen_f32_device(seed: int, stream: int, n: int, sigma: float, dst_ptr: int,
                   hip_stream: int = 0, start: int = 0) -> None:
    rc = _dev_lib().moe_gen_fill_f32_device(seed, stream, start, n, scale_for(sigma),
                                            ctypes.c_void_p(dst_ptr),
                                            ctypes.c_void_p(hip_stream))
    if rc != 0:
        raise RuntimeError(f"moe_gen_fill_f32_device failed: {rc}")


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    return (a.astype(np.uint32) << 16).view(np.float32)


# ----------------------------------------------------------------- recipes --

@dataclass(frozen=True)
class Workload:
    """One synthetic workload: layer shape, routing, value scales, seed."""
    name: str
    T: int
    d: int
    f: int
    E: int
    k: int
    sigma_w: float          # expert weights gate/up/down
    sigma_x: float = 1.0    # activations
    sigma_r: float = 0.02   # router weight
    sigma_b: float = 0.0    # per-expert router bias (0: no bias)
    e_begin: int = 0        # expert-parallel share: first local expert
    n_local: int = 0        # 0 means all experts
    n_layers: int = 1
    seed: int = 0

    @property
    def local(self) -> int:
        return self.n_local if self.n_local else self.E

    @property
    def expert_bytes(self) -> int:
        return 3 * self.d * self.f * 2

    def x(self, layer: int = 0) -> np.ndarray:
        return gen_bf16(self.seed, stream_id(KIND_X, layer), (self.T, self.d), self.sigma_x)

    def router(self, layer: int = 0) -> np.ndarray:
        return gen_f32(self.seed, stream_id(KIND_ROUTER, layer), (self.d, self.E), self.sigma_r)

    def bias(self, layer: int = 0):
        if self.sigma_b == 0.0:
            return None
        return gen_f32(self.seed, stream_id(KIND_BIAS, layer), (self.E,), self.sigma_b)

    def gate(self, e: int, layer: int = 0) -> np.ndarray:
        return gen_bf16(self.seed, stream_id(KIND_GATE, layer, e), (self.d, self.f), self.sigma_w)

    def up(self, e: int, layer: int = 0) -> np.ndarray:
        return gen_bf16(self.seed, stream_id(KIND_UP, layer, e), (self.d, self.f), self.sigma_w)

    def down(self, e: int, layer: int = 0) -> np.ndarray:
        return gen_bf16(self.seed, stream_id(KIND_DOWN, layer, e), (self.f, self.d), self.sigma_w)

    def with_(self, **kw) -> "Workload":
        from dataclasses import replace
        return replace(self, **kw)


# DBRX dimensions: Table tab:vars (D_embed 6144, D_ffn 10752), Sec. 2.1
# (16 experts, 4 selected per token).
DBRX_D = 6144
DBRX_F = 10752

WORKLOADS = {
    # small parity case: 16 tokens, d 256, 8 experts of ffn 512, top-2
    "tiny": Workload("tiny", T=16, d=256, f=512, E=8, k=2, sigma_w=0.02),
    # one decode token through the whole 16-expert layer
    "decode": Workload("decode", T=1, d=DBRX_D, f=DBRX_F, E=16, k=4, sigma_w=0.006),
    # one node's 4-of-16 expert-parallel share (experts 4s..4s+3), T in {1,4,8}
    "ep_share": Workload("ep_share", T=8, d=DBRX_D, f=DBRX_F, E=16, k=4, sigma_w=0.006,
                         e_begin=0, n_local=4),
    # prefill: 2048 tokens, N(0,1) weights and activations, skewed routing bias
    "prefill": Workload("prefill", T=2048, d=DBRX_D, f=DBRX_F, E=16, k=4, sigma_w=1.0,
                        sigma_b=1.0),
    # 32 chained layers, all 16 experts resident, 4 decode tokens
    "stack": Workload("stack", T=4, d=DBRX_D, f=DBRX_F, E=16, k=4, sigma_w=0.006,
                      n_layers=32),
}


@dataclass(frozen=True)
class AttnWorkload:
    """One synthetic self-attention workload: T new tokens at positions
    pos0 .. pos0+T-1 against a key/value cache holding positions 0 .. pos0-1.
    Shapes follow Table tab:vars (D_embed 6144, D_qkv_hidden 8192 = 48 query
    heads + 8 key + 8 value heads of 128); the head split, the rotary base and
    the norm epsilon are the readings the oracle documents."""
    name: str
    T: int
    pos0: int
    d: int
    n_heads: int
    n_kv: int
    hd: int
    max_seq: int
    theta: float = 5e5
    eps: float = 1e-5
    sigma_x: float = 1.0
    sigma_qkv: float = 0.02     # fused query/key/value projection weights
    sigma_o: float = 0.006      # output projection weights
    sigma_gamma: float = 0.1    # norm scale = 1 + N(0, sigma_gamma)
    sigma_cache: float = 1.5    # cached keys and values of earlier positions
    n_layers: int = 1
    seed: int = 0

    @property
    def nqkv(self) -> int:
        return (self.n_heads + 2 * self.n_kv) * self.hd

    def with_(self, **kw) -> "AttnWorkload":
        from dataclasses import replace
        return replace(self, **kw)

    def x(self, layer: int = 0) -> np.ndarray:
        return gen_bf16(self.seed, stream_id(KIND_ATTN_X, layer), (self.T, self.d), self.sigma_x)

    def gamma(self, layer: int = 0) -> np.ndarray:
        g = gen_f32(self.seed, stream_id(KIND_GAMMA, layer), (self.d,), self.sigma_gamma)
        return (np.float32(1.0) + g).astype(np.float32)

    def gamma2(self, layer: int = 0) -> np.ndarray:
        """The post-attention norm's scale (the MoE FFN's input norm)."""
        g = gen_f32(self.seed, stream_id(KIND_GAMMA, layer, 1), (self.d,), self.sigma_gamma)
        return (np.float32(1.0) + g).astype(np.float32)

    def wqkv(self, layer: int = 0) -> np.ndarray:
        return gen_bf16(self.seed, stream_id(KIND_WQKV, layer), (self.d, self.nqkv), self.sigma_qkv)

    def wo(self, layer: int = 0) -> np.ndarray:
        return gen_bf16(self.seed, stream_id(KIND_WO, layer), (self.n_heads * self.hd, self.d),
                        self.sigma_o)

    def cache_prefix(self, layer: int = 0):
        """Keys and values of positions 0 .. pos0-1, bf16 bits [pos0, n_kv, hd]
        (position-major)."""
        shape = (self.pos0, self.n_kv, self.hd)
        return (gen_bf16(self.seed, stream_id(KIND_KCACHE, layer), shape, self.sigma_cache),
                gen_bf16(self.seed, stream_id(KIND_VCACHE, layer), shape, self.sigma_cache))


ATTN_WORKLOADS = {
    # small parity case: 4 query heads sharing 2 key/value heads of 64, 4 new
    # tokens after 29 cached positions
    "attn_tiny": AttnWorkload("attn_tiny", T=4, pos0=29, d=256, n_heads=4, n_kv=2, hd=64,
                              max_seq=512, theta=1e4),
    # one decode token of the DBRX block after a 2047-token context (the
    # paper's long-prompt workload has 2000 input tokens)
    "attn_decode": AttnWorkload("attn_decode", T=1, pos0=2047, d=6144, n_heads=48, n_kv=8,
                                hd=128, max_seq=4096),
}
