"""MI355X-native decode attention over the DepthWeave-KV cross-depth factorized cache.

The hot path lives in ``libdwkv.so`` (hand-written HIP for gfx950, C ABI in
``include/dwkv.h``).  This package only marshals arguments: torch tensors
provide device memory and the current HIP stream.

    cache = DeviceCache(host_cache)        # upload the compressed layout
    out = cache.decode(layer)              # fp32 [B, Hq, d]
    out, err, out_ref = cache.decode(layer, probe=ProbeRef(heads, k_ref, v_ref))
    codes, offsets = cache.route(phi, u, theta)
    cache.route_range(phi, u, theta, t0, t1)      # routing of new tokens, in place
    cache.compress(layer, x_k, x_v, t0, t1)       # their Eq. 1 factors, in place
"""
from __future__ import annotations

import ctypes as C
from dataclasses import dataclass

import numpy as np

from . import binding, layout
from .binding import DwkvError, F16, BF16

__all__ = ["DeviceCache", "ProbeRef", "DwkvError", "load", "F16", "BF16", "hbm_read", "hbm_read_blocks",
           "probe_schedule"]


def load():
    return binding.load()


def _ptr(t):
    return C.c_void_p(t.data_ptr()) if t is not None else C.c_void_p(0)


def _stream(torch, device):
    return C.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def probe_schedule(step: int, period: int, n_heads: int, n_kv_heads: int, n_pos: int = 1):
    """dwkv_probe_schedule: (probed KV heads, positions) at decode step
    `step`, ([], 0) on a step that does not probe."""
    lib = load()
    heads = (C.c_int32 * max(1, n_heads))()
    npos = C.c_int32(0)
    n = lib.dwkv_probe_schedule(int(step), int(period), int(n_heads), int(n_kv_heads), int(n_pos), heads,
                                C.byref(npos))
    if n < 0:
        raise DwkvError(2, "dwkv_probe_schedule")
    return list(heads[:n]), int(npos.value)


def hbm_read_blocks() -> int:
    """Words of the sink that ``hbm_read`` writes."""
    return int(binding.load().dwkv_hbm_read_blocks())


def hbm_read(buf, sink):
    """Enqueue one read of the device tensor ``buf`` (its bytes, a multiple of
    16) on the current stream; ``sink`` is a device int32 tensor of at least
    ``hbm_read_blocks()`` elements whose xor becomes the xor of buf's 32-bit
    words.  The HBM read-stream ceiling of the device is its bytes over its
    time."""
    import torch
    lib = binding.load()
    nbytes = buf.numel() * buf.element_size()
    binding.check(lib.dwkv_hbm_read(_ptr(buf), nbytes, _ptr(sink), sink.numel(), _stream(torch, buf.device)),
                  "dwkv_hbm_read")


@dataclass
class ProbeRef:
    """Dense higher-fidelity reference cache for Eq. 3 (fp16 [n][T][d] device
    tensors).  q_prev, optional, holds the queries of earlier decode positions
    ([P-1][B][Hq][d], the decode query's dtype, slice j-1 from j steps back):
    the probe then evaluates P positions, the norms over positions and d."""
    kv_heads: list
    k_ref: object
    v_ref: object
    eps: float = 1e-6
    q_prev: object = None

    @property
    def n_pos(self) -> int:
        return 1 if self.q_prev is None else 1 + int(self.q_prev.shape[0])


class DeviceCache:
    """One factorized cache resident on the GPU in the C-ABI layout.

    ``host`` is any object carrying the layout arrays (basis, coef, rank_code,
    res_off, res_idx, res_val, res_scale, q_bits, cu_seqlens, levels, ...), for
    example a synthetic cache from ``synth.generate``."""

    def __init__(self, host, device: str = "cuda", split_tokens: int = 0):
        import torch
        self.torch = torch
        self.lib = binding.load()
        self.device = torch.device(device)
        dev = self.device
        up = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).view(dt).to(dev)
        self.basis = up(host.basis.view(np.uint16), torch.float16)
        self.coef_format = getattr(host, "coef_format", "f16")
        if self.coef_format == "int8":        # codes and their fp16 block scales
            self.coef_k = up(layout.keys_to_abi(host.coef_k.view(np.uint8), group=16), torch.uint8)
            self.coef_v = up(host.coef_v.view(np.uint8), torch.uint8)
            self.coef_scale_k = up(host.coef_scale_k.view(np.uint16), torch.float16)
            self.coef_scale_v = up(host.coef_scale_v.view(np.uint16), torch.float16)
        else:                                 # fp16: the ABI's tiled layouts
            self.coef_k = up(layout.keys_to_abi(host.coef_k.view(np.uint16)), torch.float16)
            self.coef_v = up(layout.values_to_abi(host.coef_v.view(np.uint16)), torch.float16)
            self.coef_scale_k = self.coef_scale_v = None
        self.rank_code = up(host.rank_code, torch.uint8)
        self.res_off = up(host.res_off.view(np.int32), torch.int32)
        self.res_idx = up(host.res_idx, torch.uint8)
        self.res_val = up(host.res_val, torch.uint8)
        self.res_scale = up(host.res_scale.view(np.uint16), torch.float16)
        self.q_dtype = host.q_dtype
        qdt = torch.float16 if host.q_dtype == "f16" else torch.bfloat16
        self.q = up(host.q_bits.view(np.int16), torch.int16).view(qdt)
        self.cu_host = np.ascontiguousarray(host.cu_seqlens, dtype=np.int32)
        self.cu = torch.from_numpy(self.cu_host).to(dev)
        self.batch = len(self.cu_host) - 1
        self.n_layers = host.n_layers
        self.window = host.window
        self.n_kv_heads = host.n_kv_heads
        self.n_q_heads = host.n_q_heads
        self.head_dim = host.head_dim
        self.basis_rank = host.basis_rank
        self.levels = tuple(host.levels)
        self.total_tokens = int(self.cu_host[-1])
        self.res_stride = int(host.res_stride)
        self.set_split(split_tokens)

    # -- descriptors -----------------------------------------------------------------
    def set_split(self, split_tokens: int):
        self.dims, self._cu_keep = binding.make_dims(
            batch=self.batch, n_layers=self.n_layers, window=self.window,
            n_kv_heads=self.n_kv_heads, n_q_heads=self.n_q_heads, head_dim=self.head_dim,
            basis_rank=self.basis_rank, levels=self.levels, cu_seqlens_host=self.cu_host,
            cu_seqlens_dev_ptr=self.cu.data_ptr(), total_tokens=self.total_tokens,
            res_stride=self.res_stride, split_tokens=split_tokens,
            coef_format=binding.COEF_I8 if self.coef_format == "int8" else binding.COEF_F16)
        c = binding.Cache()
        c.basis, c.rank_code = self.basis.data_ptr(), self.rank_code.data_ptr()
        c.coef_k, c.coef_v = self.coef_k.data_ptr(), self.coef_v.data_ptr()
        c.res_off, c.res_idx, c.res_val = self.res_off.data_ptr(), self.res_idx.data_ptr(), self.res_val.data_ptr()
        c.res_scale = self.res_scale.data_ptr()
        if self.coef_scale_k is not None:
            c.coef_k_scale, c.coef_v_scale = self.coef_scale_k.data_ptr(), self.coef_scale_v.data_ptr()
        self.cstruct = c
        self._ws = {}

    @property
    def split_tokens(self) -> int:
        return int(self.lib.dwkv_split_tokens(C.byref(self.dims)))

    @property
    def uses_token_lane(self) -> bool:
        """True when dwkv_decode runs the token-lane split kernel for this cache."""
        return int(self.lib.dwkv_decode_kernel(C.byref(self.dims))) == 1

    @property
    def decode_launches(self) -> int:
        """Kernel launches of one decode call without a probe (the split-K pass and the merge)."""
        return int(self.lib.dwkv_decode_launches(C.byref(self.dims), None))

    def _probe_struct(self, probe: ProbeRef | None, err, out_ref):
        if probe is None:
            return None, None
        heads = np.ascontiguousarray(probe.kv_heads, dtype=np.int32)
        p = binding.Probe()
        p.n_heads = len(heads)
        p.kv_heads_host = heads.ctypes.data_as(C.POINTER(C.c_int32))
        p.k_ref, p.v_ref = probe.k_ref.data_ptr(), probe.v_ref.data_ptr()
        p.eps = probe.eps
        p.err = err.data_ptr()
        p.out_ref = out_ref.data_ptr() if out_ref is not None else None
        p.n_pos = probe.n_pos
        if probe.q_prev is not None:
            qp = probe.q_prev
            if tuple(qp.shape[1:]) != (self.batch, self.n_q_heads, self.head_dim) or not qp.is_contiguous():
                raise ValueError("q_prev must be a contiguous [P-1, B, Hq, d] tensor")
            p.q_prev = qp.data_ptr()
        return p, heads

    def workspace_bytes(self, probe: ProbeRef | None = None) -> int:
        torch = self.torch
        G = self.n_q_heads // self.n_kv_heads
        err = torch.empty(1, device=self.device)
        p, keep = self._probe_struct(probe, err, None)
        n = self.lib.dwkv_workspace_bytes(C.byref(self.dims), C.byref(p) if p is not None else None)
        if n == 0:
            raise DwkvError(2, "dwkv_workspace_bytes")
        return int(n)

    def new_workspace(self, probe: ProbeRef | None = None):
        """A fresh decode workspace (zero-filled; the library needs no initial contents)."""
        return self.torch.zeros(self.workspace_bytes(probe), dtype=self.torch.uint8, device=self.device)

    def workspace(self, probe: ProbeRef | None = None):
        """A decode workspace, allocated once per probe shape and reused."""
        need = self.workspace_bytes(probe)
        key = None if probe is None else (len(probe.kv_heads), probe.n_pos)
        ws = self._ws.get(key)
        if ws is None or ws.numel() < need:
            ws = self.new_workspace(probe)
            self._ws[key] = ws
        return ws

    # -- calls -----------------------------------------------------------------------
    def decode(self, layer: int, q=None, sm_scale: float | None = None, probe: ProbeRef | None = None,
               out=None, workspace=None, with_ref: bool = True, err=None):
        """Per-layer decode attention; returns out [B,Hq,d] fp32, or
        (out, err [B, n*G], out_ref [B, n*G, d]) with a probe (err may be given)."""
        torch = self.torch
        if q is None:
            q = self.q[layer]
        qt = F16 if q.dtype == torch.float16 else BF16
        if q.dtype not in (torch.float16, torch.bfloat16):
            raise TypeError("q must be float16 or bfloat16")
        B, Hq, d = self.batch, self.n_q_heads, self.head_dim
        if out is None:
            out = torch.empty((B, Hq, d), dtype=torch.float32, device=self.device)
        G = Hq // self.n_kv_heads
        out_ref = None
        if probe is not None:
            if probe.q_prev is not None and probe.q_prev.dtype != q.dtype:
                raise TypeError("q_prev must have the decode query's dtype")
            n = len(probe.kv_heads)
            if err is None:
                err = torch.empty((B, n * G), dtype=torch.float32, device=self.device)
            out_ref = torch.empty((B, n * G, d), dtype=torch.float32, device=self.device) if with_ref else None
        p, keep = self._probe_struct(probe, err, out_ref)
        ws = workspace if workspace is not None else self.workspace(probe)
        st = self.lib.dwkv_decode(C.byref(self.dims), C.byref(self.cstruct), int(layer), _ptr(q), qt,
                                  float(sm_scale or 0.0), _ptr(out), C.byref(p) if p is not None else None,
                                  _ptr(ws), ws.numel(), _stream(torch, self.device))
        binding.check(st, "dwkv_decode")
        return out if probe is None else (out, err, out_ref)

    def decode_noalloc(self, layer: int, q=None, sm_scale: float | None = None, out=None,
                       probe: ProbeRef | None = None, err=None):
        """dwkv_decode_noalloc: decode with the library's static scratch (no
        workspace); out [B,Hq,d] fp32 (and err [B, n*G] with a probe) must be
        given or are allocated here by torch.  Returns out, or (out, err)."""
        torch = self.torch
        if q is None:
            q = self.q[layer]
        if q.dtype not in (torch.float16, torch.bfloat16):
            raise TypeError("q must be float16 or bfloat16")
        qt = F16 if q.dtype == torch.float16 else BF16
        if out is None:
            out = torch.empty((self.batch, self.n_q_heads, self.head_dim), dtype=torch.float32, device=self.device)
        if probe is not None and err is None:
            G = self.n_q_heads // self.n_kv_heads
            err = torch.empty((self.batch, len(probe.kv_heads) * G), dtype=torch.float32, device=self.device)
        p, keep = self._probe_struct(probe, err, None)
        st = self.lib.dwkv_decode_noalloc(C.byref(self.dims), C.byref(self.cstruct), int(layer), _ptr(q), qt,
                                          float(sm_scale or 0.0), _ptr(out), C.byref(p) if p is not None else None,
                                          _stream(torch, self.device))
        binding.check(st, "dwkv_decode_noalloc")
        return out if probe is None else (out, err)

    def decode_partials(self, layer: int, q=None, sm_scale: float | None = None, workspace=None,
                        probe: ProbeRef | None = None, err=None):
        """First half of decode: the split-K pass(es); dwkv_decode_merge finishes it
        (with the same probe and err)."""
        torch = self.torch
        if q is None:
            q = self.q[layer]
        qt = F16 if q.dtype == torch.float16 else BF16
        p, keep = self._probe_struct(probe, err, None)
        ws = workspace if workspace is not None else self.workspace(probe)
        st = self.lib.dwkv_decode_partials(C.byref(self.dims), C.byref(self.cstruct), int(layer), _ptr(q), qt,
                                           float(sm_scale or 0.0), C.byref(p) if p is not None else None,
                                           _ptr(ws), ws.numel(), _stream(torch, self.device))
        binding.check(st, "dwkv_decode_partials")

    def decode_merge(self, layer: int, out=None, workspace=None, probe: ProbeRef | None = None, err=None):
        """Second half of decode: merges the split partials of `layer` into out [B,Hq,d]
        (and, with a probe, writes err [B, n*G])."""
        torch = self.torch
        if out is None:
            out = torch.empty((self.batch, self.n_q_heads, self.head_dim), dtype=torch.float32, device=self.device)
        p, keep = self._probe_struct(probe, err, None)
        ws = workspace if workspace is not None else self.workspace(probe)
        st = self.lib.dwkv_decode_merge(C.byref(self.dims), C.byref(self.cstruct), int(layer), _ptr(out),
                                        C.byref(p) if p is not None else None, _ptr(ws), ws.numel(),
                                        _stream(torch, self.device))
        binding.check(st, "dwkv_decode_merge")
        return out

    def probe_feature(self, layer: int, kv_heads, err, phi, fresh: bool):
        """dwkv_probe_feature: fold one probed layer's Eq. 3 errors err [B, n*G]
        into column 3 of the layer's window of phi [M, Hkv, T, 4] (in place)."""
        heads = np.ascontiguousarray(kv_heads, dtype=np.int32)
        st = self.lib.dwkv_probe_feature(C.byref(self.dims), int(layer), len(heads),
                                         heads.ctypes.data_as(C.POINTER(C.c_int32)), _ptr(err), int(bool(fresh)),
                                         _ptr(phi), _stream(self.torch, self.device))
        binding.check(st, "dwkv_probe_feature")
        return phi

    def route(self, phi, u, theta, rank_code=None, res_off=None):
        """Eq. 2 routing on the GPU; returns (rank_code uint8 [M,Hkv,T], res_off int32-view [M,Hkv,T+1])."""
        torch = self.torch
        M, Hk, T = self.n_layers // self.window, self.n_kv_heads, self.total_tokens
        if rank_code is None:
            rank_code = torch.empty((M, Hk, T), dtype=torch.uint8, device=self.device)
        if res_off is None:
            res_off = torch.empty((M, Hk, T + 1), dtype=torch.int32, device=self.device)
        need = self.lib.dwkv_route_workspace_bytes(C.byref(self.dims))
        ws = torch.empty(max(int(need), 1), dtype=torch.uint8, device=self.device)
        st = self.lib.dwkv_route(C.byref(self.dims), _ptr(phi), _ptr(u), _ptr(theta), _ptr(rank_code),
                                 _ptr(res_off), _ptr(ws), ws.numel(), _stream(torch, self.device))
        binding.check(st, "dwkv_route")
        return rank_code, res_off

    def route_range(self, phi, u, theta, t0: int, t1: int, rank_code=None, res_off=None):
        """Eq. 2 routing of packed tokens [t0, t1), continuing the offset table in
        place (by default the cache's own rank_code / res_off)."""
        torch = self.torch
        rank_code = self.rank_code if rank_code is None else rank_code
        res_off = self.res_off if res_off is None else res_off
        need = self.lib.dwkv_route_workspace_bytes(C.byref(self.dims))
        ws = torch.empty(max(int(need), 1), dtype=torch.uint8, device=self.device)
        st = self.lib.dwkv_route_range(C.byref(self.dims), _ptr(phi), _ptr(u), _ptr(theta), int(t0), int(t1),
                                       _ptr(rank_code), _ptr(res_off), _ptr(ws), ws.numel(),
                                       _stream(torch, self.device))
        binding.check(st, "dwkv_route_range")
        return rank_code, res_off

    def route_budget(self, phi, u, entries, t0: int, t1: int, rank_code=None, res_off=None):
        """Two-level Eq. 2 routing of tokens [t0, t1) under a budget of entries
        (int64 [M, Hkv], device) per (window, head); in place by default."""
        torch = self.torch
        rank_code = self.rank_code if rank_code is None else rank_code
        res_off = self.res_off if res_off is None else res_off
        need = int(self.lib.dwkv_route_budget_workspace_bytes(C.byref(self.dims)))
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        st = self.lib.dwkv_route_budget(C.byref(self.dims), _ptr(phi), _ptr(u), _ptr(entries), int(t0), int(t1),
                                        _ptr(rank_code), _ptr(res_off), _ptr(ws), ws.numel(),
                                        _stream(torch, self.device))
        binding.check(st, "dwkv_route_budget")
        return rank_code, res_off

    def compress(self, layer: int, x_k, x_v, t0: int, t1: int, gate=None):
        """Append/compress packed tokens [t0, t1) of `layer` in place from dense
        fp16 keys / values x_k, x_v [t1-t0, Hkv, d]; gate: None or fp32 [2, Hkv, t1-t0]."""
        torch = self.torch
        for x in (x_k, x_v):
            if x.dtype != torch.float16 or not x.is_contiguous():
                raise TypeError("x_k / x_v must be contiguous float16")
        if gate is not None and (gate.dtype != torch.float32 or not gate.is_contiguous()):
            raise TypeError("gate must be contiguous float32")
        st = self.lib.dwkv_compress(C.byref(self.dims), C.byref(self.cstruct), int(layer), _ptr(x_k), _ptr(x_v),
                                    _ptr(gate), int(t0), int(t1), _stream(torch, self.device))
        binding.check(st, "dwkv_compress")

    @property
    def decode_append_launches(self) -> int:
        return int(self.lib.dwkv_decode_append_launches(C.byref(self.dims)))

    def decode_append(self, layer: int, x_k, x_v, gate=None, q=None, sm_scale: float | None = None, out=None,
                      workspace=None):
        """dwkv_decode_append: append the new token of every sequence (its
        last) from x_k, x_v [B, Hkv, d] fp16 (gate None or fp32 [2, Hkv, B]),
        then decode the layer; returns out [B, Hq, d] fp32."""
        torch = self.torch
        for x in (x_k, x_v):
            if x.dtype != torch.float16 or not x.is_contiguous():
                raise TypeError("x_k / x_v must be contiguous float16")
        if gate is not None and (gate.dtype != torch.float32 or not gate.is_contiguous()):
            raise TypeError("gate must be contiguous float32")
        if q is None:
            q = self.q[layer]
        if q.dtype not in (torch.float16, torch.bfloat16):
            raise TypeError("q must be float16 or bfloat16")
        qt = F16 if q.dtype == torch.float16 else BF16
        if out is None:
            out = torch.empty((self.batch, self.n_q_heads, self.head_dim), dtype=torch.float32, device=self.device)
        need = int(self.lib.dwkv_decode_append_workspace_bytes(C.byref(self.dims)))
        if need == 0:
            raise DwkvError(2, "dwkv_decode_append_workspace_bytes")
        if workspace is None:
            ws = self._ws.get("append")
            if ws is None or ws.numel() < need:
                ws = torch.zeros(need, dtype=torch.uint8, device=self.device)
                self._ws["append"] = ws
            workspace = ws
        st = self.lib.dwkv_decode_append(C.byref(self.dims), C.byref(self.cstruct), int(layer), _ptr(q), qt,
                                         float(sm_scale or 0.0), _ptr(out), _ptr(x_k), _ptr(x_v), _ptr(gate),
                                         _ptr(workspace), workspace.numel(), _stream(torch, self.device))
        binding.check(st, "dwkv_decode_append")
        return out

    def decode_features(self, layer: int, phi, q=None, sm_scale: float | None = None, out=None, workspace=None):
        """dwkv_decode plus the router's attention features: phi fp32 [M, Hkv, T, 4]
        (columns 0 mass, 1 spike) is updated in place; returns out [B, Hq, d]."""
        torch = self.torch
        if q is None:
            q = self.q[layer]
        qt = F16 if q.dtype == torch.float16 else BF16
        if out is None:
            out = torch.empty((self.batch, self.n_q_heads, self.head_dim), dtype=torch.float32, device=self.device)
        if workspace is None:
            n = int(self.lib.dwkv_features_workspace_bytes(C.byref(self.dims)))
            if n == 0:
                raise DwkvError(3, "dwkv_features_workspace_bytes")
            workspace = torch.empty(n, dtype=torch.uint8, device=self.device)
        st = self.lib.dwkv_decode_features(C.byref(self.dims), C.byref(self.cstruct), int(layer), _ptr(q), qt,
                                           float(sm_scale or 0.0), _ptr(out), _ptr(phi), _ptr(workspace),
                                           workspace.numel(), _stream(torch, self.device))
        binding.check(st, "dwkv_decode_features")
        return out

    def sketch_basis(self, window: int, seq: int, x, omega):
        """Randomized-sketch bases of (seq, window) from its prefill x fp16
        [w, 2, n, Hkv, d] and sketch matrix omega fp16 [w*n, r_b]; in place."""
        torch = self.torch
        n = int(x.shape[2])
        need = int(self.lib.dwkv_sketch_workspace_bytes(C.byref(self.dims), n))
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        st = self.lib.dwkv_sketch_basis(C.byref(self.dims), C.byref(self.cstruct), int(window), int(seq), _ptr(x),
                                        _ptr(omega), n, _ptr(ws), ws.numel(), _stream(torch, self.device))
        binding.check(st, "dwkv_sketch_basis")

    def materialize(self, layer: int, k_out=None, v_out=None):
        """Eq. 1 written out for `layer`: K_hat fp16 [Hkv, T, d] and V_hat fp16
        [Hkv, T16/16, d, 16] (the blocked layout of the dense decode)."""
        torch = self.torch
        Hk, T, d = self.n_kv_heads, self.total_tokens, self.head_dim
        T16 = -(-T // 16) * 16
        if k_out is None:
            k_out = torch.empty((Hk, T, d), dtype=torch.float16, device=self.device)
        if v_out is None:
            v_out = torch.empty((Hk, T16 // 16, d, 16), dtype=torch.float16, device=self.device)
        st = self.lib.dwkv_materialize(C.byref(self.dims), C.byref(self.cstruct), int(layer), _ptr(k_out),
                                       _ptr(v_out), _stream(torch, self.device))
        binding.check(st, "dwkv_materialize")
        return k_out, v_out

    def dense_decode(self, k, v, q, sm_scale: float | None = None, out=None, workspace=None):
        """Decode attention over a dense fp16 cache k [Hkv, T, d], v [Hkv, T16/16, d, 16]."""
        torch = self.torch
        qt = F16 if q.dtype == torch.float16 else BF16
        if out is None:
            out = torch.empty((self.batch, self.n_q_heads, self.head_dim), dtype=torch.float32, device=self.device)
        if workspace is None:
            workspace = torch.empty(int(self.lib.dwkv_dense_workspace_bytes(C.byref(self.dims))),
                                    dtype=torch.uint8, device=self.device)
        st = self.lib.dwkv_dense_decode(C.byref(self.dims), _ptr(k), _ptr(v), _ptr(q), qt, float(sm_scale or 0.0),
                                        _ptr(out), _ptr(workspace), workspace.numel(),
                                        _stream(torch, self.device))
        binding.check(st, "dwkv_dense_decode")
        return out

    def residual_map(self, layer: int, z: int, kv_head: int, t0: int, t1: int):
        torch = self.torch
        dense = torch.empty((max(t1 - t0, 0), self.head_dim), dtype=torch.float32, device=self.device)
        st = self.lib.dwkv_residual_map(C.byref(self.dims), C.byref(self.cstruct), int(layer), int(z),
                                        int(kv_head), int(t0), int(t1), _ptr(dense),
                                        _stream(torch, self.device))
        binding.check(st, "dwkv_residual_map")
        return dense

    def coef_host(self):
        """The device coefficients in the host layout (fp16 as uint16): keys
        [L][Hkv][T][r_b], values [L][Hkv][T16/16][r_b][16] (int8: codes, same shapes)."""
        k = self.coef_k.cpu().numpy()
        v = self.coef_v.cpu().numpy()
        L, Hk, T, rb = self.n_layers, self.n_kv_heads, self.total_tokens, self.basis_rank
        T16 = -(-T // 16) * 16
        if self.coef_format == "int8":
            return layout.keys_from_abi(k.reshape(L, Hk, T16 // 16, rb // 16, 16, 16), T), v
        k, v = k.view(np.uint16), v.view(np.uint16)
        keys = layout.keys_from_abi(k.reshape(L, Hk, T16 // 16, rb // 8, 16, 8), T)
        vals = layout.values_from_abi(v.reshape(L, Hk, T16 // 8, rb, 8))
        return keys, vals

    def validate(self):
        """Returns (ok, bad_index); raises on argument errors."""
        torch = self.torch
        ws = torch.empty(int(self.lib.dwkv_validate_workspace_bytes()), dtype=torch.uint8, device=self.device)
        bad = C.c_int64(-1)
        st = self.lib.dwkv_validate(C.byref(self.dims), C.byref(self.cstruct), C.byref(bad), _ptr(ws),
                                    ws.numel(), _stream(torch, self.device))
        if st == 5:
            return False, int(bad.value)
        binding.check(st, "dwkv_validate")
        return True, -1
