"""ctypes binding of libmxmoe.so (C ABI in include/mxmoe.h).

Argument marshalling only: every step of the forward runs in the library's HIP
kernels.  PyTorch provides device memory and the current stream.  There is no
fallback: if the library is missing or a call fails, an exception is raised.
"""

from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmxmoe.so")

F16, BF16 = 0, 1
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)


class Scheme_t(C.Structure):
    _fields_ = [("w_bits", C.c_int32), ("a_bits", C.c_int32), ("w_group", C.c_int32),
                ("a_group", C.c_int32), ("symmetric", C.c_int32), ("fmt", C.c_int32)]


class Linear_t(C.Structure):
    _fields_ = [("n", C.c_int32), ("k", C.c_int32), ("s", Scheme_t)]


class Block_t(C.Structure):
    _fields_ = [("hidden", C.c_int32), ("ffn", C.c_int32), ("n_experts", C.c_int32),
                ("top_k", C.c_int32), ("n_shared", C.c_int32), ("ffn_shared", C.c_int32),
                ("act", C.c_int), ("scheme", C.POINTER(Scheme_t)), ("packed", C.POINTER(C.c_void_p))]


N_PHASES = 5
PHASE_NAMES = ("route_plan_xquant", "gemm_gate_up", "hquant", "gemm_down", "combine")


class ForwardOpts_t(C.Structure):
    _fields_ = [("expert_mask", C.POINTER(C.c_uint8)), ("reserved0", C.c_int32),
                ("skip_combine", C.c_int32), ("events", C.POINTER(C.c_void_p)),
                ("router_logits", C.c_void_p), ("renormalize", C.c_int32), ("shared_logits", C.c_void_p),
                ("shared_w", C.c_void_p), ("fp32_slots", C.c_int32), ("reserved1", C.c_int32)]


WS_FIELDS = ["status", "counts", "offsets", "sorted_pair", "inv", "plan", "xq8", "xs8", "xq4", "xs4",
             "h", "h_shared", "hq", "hs", "hq_shared", "hs_shared", "slots", "total", "plan_queue_cap",
             "plan_flat_cap", "partial", "partial_floats", "rsx", "rsh", "rsh_shared", "xq4g", "xs4g", "hsg",
             "hsg_shared", "xqmx", "xsmx", "hqmx", "hsmx", "hqmx_shared", "hsmx_shared", "router_ids", "router_w",
             "shared_w", "xqf8", "xsf8", "xqf6", "xsf6"]


class WsLayout_t(C.Structure):
    _fields_ = [(f, C.c_size_t) for f in WS_FIELDS]


EXPORTS = [
    "mxmoe_packed_bytes", "mxmoe_pack_weights", "mxmoe_unpack_weights", "mxmoe_route_workspace_bytes",
    "mxmoe_route_permute", "mxmoe_router_topk", "mxmoe_act_quant", "mxmoe_linear_workspace_bytes", "mxmoe_linear_forward",
    "mxmoe_block_table_bytes", "mxmoe_block_table_fill", "mxmoe_workspace_bytes", "mxmoe_moe_forward",
    "mxmoe_moe_forward_ex", "mxmoe_workspace_layout", "mxmoe_status_string", "mxmoe_version",
    "mxmoe_moe_forward_noalloc", "mxmoe_set_tile_costs", "mxmoe_get_tile_costs",
]
TILE_COST_SHAPE = (2, 11, 4, 4)     # [phase][scheme][configuration][a, bs, bu, h], MXMOE_TILE_COST_ENTRIES
NOALLOC_SCRATCH_BYTES = 128 << 20   # MXMOE_NOALLOC_SCRATCH_BYTES

_lib = None


def load_library(path: str = LIB_PATH) -> C.CDLL:
    """Load libmxmoe.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2505_05799_amd.build`")
    lib = C.CDLL(path)
    vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    PL, PB = C.POINTER(Linear_t), C.POINTER(Block_t)
    sig = {
        "mxmoe_packed_bytes": (sz, [PL, C.c_int]),
        "mxmoe_pack_weights": (C.c_int, [PL, C.c_int, C.c_int, vp, vp, vp, vp, sz, vp]),
        "mxmoe_unpack_weights": (C.c_int, [PL, C.c_int, vp, vp, vp, vp, vp]),
        "mxmoe_route_workspace_bytes": (sz, [i32, i32, i32]),
        "mxmoe_route_permute": (C.c_int, [vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, sz, vp]),
        "mxmoe_router_topk": (C.c_int, [vp, i32, i32, i32, i32, vp, i32, vp, vp, vp, vp]),
        "mxmoe_act_quant": (C.c_int, [vp, C.c_int, i32, i32, i64, i32, vp, vp, vp]),
        "mxmoe_linear_workspace_bytes": (sz, [PL, i32]),
        "mxmoe_linear_forward": (C.c_int, [PL, C.c_int, vp, i32, vp, vp, vp, sz, vp]),
        "mxmoe_block_table_bytes": (sz, [PB]),
        "mxmoe_block_table_fill": (C.c_int, [PB, vp, sz]),
        "mxmoe_workspace_bytes": (sz, [PB, i32]),
        "mxmoe_moe_forward": (C.c_int, [PB, vp, i32, vp, vp, vp, vp, vp, sz, vp]),
        "mxmoe_moe_forward_ex": (C.c_int, [PB, vp, i32, vp, vp, vp, vp, vp, sz,
                                           C.POINTER(ForwardOpts_t), vp]),
        "mxmoe_workspace_layout": (C.c_int, [PB, i32, C.POINTER(WsLayout_t)]),
        "mxmoe_moe_forward_noalloc": (C.c_int, [PB, vp, i32, vp, vp, vp, vp, vp]),
        "mxmoe_status_string": (C.c_char_p, [C.c_int]),
        "mxmoe_version": (i32, []),
        "mxmoe_set_tile_costs": (C.c_int, [vp, i32]),
        "mxmoe_get_tile_costs": (C.c_int, [vp, i32]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    # the run-time plan prices tiles with the profiled cost table when there is one
    from . import tile_cost
    if os.path.exists(tile_cost.DEFAULT_TABLE):
        set_tile_costs(tile_cost.CostTable.load().device_table())
    return lib


def set_tile_costs(table=None):
    """Install the run-time plan's tile cost table (int32 TILE_COST_SHAPE, ps),
    or the library's roofline default with None (mxmoe_set_tile_costs)."""
    lib = load_library()
    if table is None:
        _check(lib.mxmoe_set_tile_costs(None, 0), "mxmoe_set_tile_costs")
        return
    t = np.ascontiguousarray(table, dtype=np.int32)
    if t.shape != TILE_COST_SHAPE:
        raise ValueError(f"tile cost table of shape {t.shape}, expected {TILE_COST_SHAPE}")
    _check(lib.mxmoe_set_tile_costs(t.ctypes.data_as(C.c_void_p), t.size), "mxmoe_set_tile_costs")


def get_tile_costs() -> np.ndarray:
    """The tile cost table forwards use now (mxmoe_get_tile_costs)."""
    t = np.zeros(TILE_COST_SHAPE, dtype=np.int32)
    _check(load_library().mxmoe_get_tile_costs(t.ctypes.data_as(C.c_void_p), t.size), "mxmoe_get_tile_costs")
    return t


class MxmoeError(RuntimeError):
    def __init__(self, status: int, what: str):
        lib = load_library()
        super().__init__(f"{what}: {lib.mxmoe_status_string(status).decode()} (status {status})")
        self.status = status


def _check(status: int, what: str):
    if status != OK:
        raise MxmoeError(status, what)


def _torch():
    import torch
    return torch


def _stream_ptr(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _ptr(t) -> C.c_void_p:
    return C.c_void_p(0 if t is None else t.data_ptr())


def scheme_t(s) -> Scheme_t:
    return Scheme_t(s.w_bits, s.a_bits, s.w_group, s.a_group, s.symmetric, getattr(s, "fmt", 0))


def act_code(act: str) -> int:
    return {"fp16": F16, "bf16": BF16}[act]


def _dev(arr: np.ndarray, device):
    """numpy -> device tensor with the same bytes (16-bit data travels as int16);
    a torch tensor is moved as it is."""
    torch = _torch()
    if isinstance(arr, torch.Tensor):
        return arr.contiguous().to(device)
    a = np.ascontiguousarray(arr)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    if a.dtype == np.float16:
        a = a.view(np.int16)
    return torch.from_numpy(a.copy()).to(device)


def act_tensor(x: np.ndarray, act: str, device="cuda"):
    """numpy activation storage (float16 or bf16 bits) -> torch tensor of the act dtype."""
    torch = _torch()
    t = _dev(x, device)
    return t.view(torch.float16 if act == "fp16" else torch.bfloat16)


def act_numpy(t, act: str) -> np.ndarray:
    """torch act tensor -> numpy storage (float16 array or bf16 bits)."""
    torch = _torch()
    a = t.detach().contiguous().view(torch.int16).cpu().numpy()
    return a.view(np.float16) if act == "fp16" else a.view(np.uint16)


def empty_aligned(nbytes: int, device="cuda"):
    torch = _torch()
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# --------------------------------------------------------------- packing
def operand_bytes(scheme, n: int, k: int):
    """Bytes the packer reads from (codes, scales, zeros) for a scheme (None: not read)."""
    s = scheme
    if s.w_bits == 16:
        return 2 * n * k, None, None
    if getattr(s, "fmt", 0) == 1:
        return n * k, n * (k // 32), None
    if s.a_bits == 16:
        return n * k, 2 * n * (k // 128), 2 * n * (k // 128)
    if s.w_group > 0:
        return n * k, 2 * n * (k // 128), None
    return n * k, 4 * n, None


def _nbytes(arr) -> int:
    if arr is None:
        return 0
    if hasattr(arr, "element_size"):
        return arr.numel() * arr.element_size()
    return np.asarray(arr).nbytes


def check_operands(q):
    """Raise ValueError unless the codes / scales / zeros of a QLinear hold at
    least the bytes the packer reads for its scheme (the packer takes raw
    pointers and cannot check their extent)."""
    want = operand_bytes(q.scheme, q.n, q.k)
    for name, arr, need in zip(("codes", "scales", "zeros"), (q.codes, q.scales, q.zeros), want):
        if need is not None and (arr is None or _nbytes(arr) < need):
            raise ValueError(f"{q.scheme.name} {q.n}x{q.k}: {name} hold {_nbytes(arr)} bytes, the packer reads {need}")


class PackedLinear:
    """One linear packed on the device (owns the packed buffer)."""

    def __init__(self, q, act: str, device="cuda", stream=None):
        lib = load_library()
        check_operands(q)
        self.q = q
        self.act = act
        self.L = Linear_t(q.n, q.k, scheme_t(q.scheme))
        nbytes = lib.mxmoe_packed_bytes(C.byref(self.L), act_code(act))
        if nbytes == 0:
            raise MxmoeError(ERR_UNSUPPORTED, f"packed_bytes({q.scheme.name} {q.n}x{q.k})")
        self.nbytes = nbytes
        self.buf = empty_aligned(nbytes, device)
        codes = _dev(q.codes, device)
        scales = _dev(q.scales, device) if q.scales is not None else None
        zeros = _dev(q.zeros, device) if q.zeros is not None else None
        _check(lib.mxmoe_pack_weights(C.byref(self.L), act_code(act), BF16, _ptr(codes), _ptr(scales),
                                      _ptr(zeros), _ptr(self.buf), nbytes, _stream_ptr(stream)),
               "mxmoe_pack_weights")
        self._keep = (codes, scales, zeros)   # alive until the pack kernel has run

    def release_sources(self):
        self._keep = None

    def unpack(self, stream=None):
        """Device unpack -> (codes, scales, zeros) as numpy arrays."""
        torch = _torch()
        lib = load_library()
        q = self.q
        s = q.scheme
        if s.w_bits == 16:
            codes = torch.empty((q.n, q.k), dtype=torch.int16, device=self.buf.device)
        else:
            codes = torch.empty((q.n, q.k), dtype=torch.uint8, device=self.buf.device)
        scales = zeros = None
        if s.w_bits < 16 and s.a_bits == 16:
            scales = torch.empty((q.n, q.k // 128), dtype=torch.int16, device=self.buf.device)
            zeros = torch.empty_like(scales)
        elif s.fmt == 1:                          # mxfp4: E8M0 bytes per 32
            scales = torch.empty((q.n, q.k // 32), dtype=torch.uint8, device=self.buf.device)
        elif s.w_bits < 16 and s.w_group > 0:     # w4a4-g128: fp16 group scales
            scales = torch.empty((q.n, q.k // 128), dtype=torch.int16, device=self.buf.device)
        elif s.w_bits < 16:
            scales = torch.empty(q.n, dtype=torch.float32, device=self.buf.device)
        _check(lib.mxmoe_unpack_weights(C.byref(self.L), act_code(self.act), _ptr(self.buf), _ptr(codes),
                                        _ptr(scales), _ptr(zeros), _stream_ptr(stream)),
               "mxmoe_unpack_weights")
        torch.cuda.synchronize()
        c = codes.cpu().numpy()
        if s.w_bits == 16:
            c = c.view(np.uint16)
        elif s.a_bits < 16 and s.fmt in (0, 3):
            c = c.view(np.int8)
        sc = None if scales is None else scales.cpu().numpy()
        if sc is not None and s.fmt == 0 and (s.a_bits == 16 or s.w_group > 0):
            sc = sc.view(np.float16)
        z = None if zeros is None else zeros.cpu().numpy().view(np.float16)
        return c, sc, z


def linear_forward(pl: PackedLinear, a, stream=None, return_ws: bool = False):
    """out = a W^T through the micro-kernels: int32 for w8a8/w4a4 (per channel,
    int8 or FP6 operands), else fp32 (fp8: scaled by s_a[m] s_w[n]).  return_ws: also return the
    workspace (its tile plan starts at offset 0)."""
    torch = _torch()
    lib = load_library()
    m = a.shape[0]
    s = pl.q.scheme
    raw_int = s.a_bits < 16 and s.a_group < 0 and getattr(s, "fmt", 0) in (0, 3)
    out = torch.empty((m, pl.q.n), dtype=torch.int32 if raw_int else torch.float32, device=a.device)
    wsb = lib.mxmoe_linear_workspace_bytes(C.byref(pl.L), m)
    ws = empty_aligned(wsb, a.device)
    _check(lib.mxmoe_linear_forward(C.byref(pl.L), act_code(pl.act), _ptr(pl.buf), m, _ptr(a.contiguous()),
                                    _ptr(out), _ptr(ws), wsb, _stream_ptr(stream)), "mxmoe_linear_forward")
    return (out, ws) if return_ws else out


# --------------------------------------------------------------- routing
def route_permute(topk_ids, E: int, stream=None):
    torch = _torch()
    lib = load_library()
    T, k = topk_ids.shape
    dev = topk_ids.device
    counts = torch.empty(E, dtype=torch.int32, device=dev)
    offsets = torch.empty(E + 1, dtype=torch.int32, device=dev)
    sp = torch.full((max(T * k, 1),), -7, dtype=torch.int32, device=dev)
    inv = torch.empty(max(T * k, 1), dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    wsb = lib.mxmoe_route_workspace_bytes(T, k, E)
    ws = empty_aligned(wsb, dev)
    _check(lib.mxmoe_route_permute(_ptr(topk_ids.contiguous()), T, k, E, _ptr(counts), _ptr(offsets), _ptr(sp),
                                   _ptr(inv), _ptr(status), _ptr(ws), wsb, _stream_ptr(stream)),
           "mxmoe_route_permute")
    return {"counts": counts, "offsets": offsets, "sorted_pair": sp[: T * k], "inv": inv[: T * k],
            "status": status}


def router_topk(logits, k: int, renormalize: bool = False, shared_logits=None, stream=None):
    """Router front-end: (ids int32 [T,k], weights fp32 [T,k], shared gates fp32
    [T,n_shared] or None) from fp32 logits [T,E] (and shared-gate logits)."""
    torch = _torch()
    lib = load_library()
    T, E = logits.shape
    ids = torch.empty((T, k), dtype=torch.int32, device=logits.device)
    w = torch.empty((T, k), dtype=torch.float32, device=logits.device)
    n_sh = 0 if shared_logits is None else shared_logits.shape[1]
    shw = None if shared_logits is None else torch.empty((T, n_sh), dtype=torch.float32, device=logits.device)
    _check(lib.mxmoe_router_topk(_ptr(logits), T, E, k, 1 if renormalize else 0, _ptr(shared_logits), n_sh, _ptr(ids),
                                 _ptr(w), _ptr(shw), _stream_ptr(stream)), "mxmoe_router_topk")
    return ids, w, shw


def act_quant(a, act: str, qmax: int, stream=None):
    torch = _torch()
    lib = load_library()
    rows, cols = a.shape
    codes = torch.empty((rows, cols), dtype=torch.int8, device=a.device)
    scales = torch.empty(rows, dtype=torch.float32, device=a.device)
    _check(lib.mxmoe_act_quant(_ptr(a), act_code(act), rows, cols, a.stride(0), qmax, _ptr(codes), _ptr(scales),
                               _stream_ptr(stream)), "mxmoe_act_quant")
    return codes, scales


# --------------------------------------------------------------- block
class MoEBlock:
    """A packed MoE block on one GPU: weights, block table and workspace."""

    def __init__(self, block, device="cuda", T_max: Optional[int] = None, stream=None,
                 packed: Optional[List[List[PackedLinear]]] = None):
        """`packed`: already packed linears per expert (may repeat objects) instead
        of packing block.linears."""
        torch = _torch()
        lib = load_library()
        cfg = block.cfg
        self.cfg = cfg
        self.act = cfg.act
        self.device = device
        self.packed: List[List[PackedLinear]] = [list(ps) for ps in packed] if packed is not None else []
        if packed is None:
            for lins in block.linears:
                self.packed.append([PackedLinear(q, cfg.act, device, stream) for q in lins])
        G = cfg.E + cfg.n_shared
        if len(self.packed) != G:
            raise ValueError(f"{len(self.packed)} packed experts for a block of {G}")
        self._schemes = (Scheme_t * (3 * G))(*[scheme_t(p.q.scheme) for ps in self.packed for p in ps])
        self._ptrs = (C.c_void_p * (3 * G))(*[p.buf.data_ptr() for ps in self.packed for p in ps])
        self.B = Block_t(cfg.H, cfg.F, cfg.E, cfg.k, cfg.n_shared, cfg.F_shared if cfg.n_shared else 0,
                         act_code(cfg.act), C.cast(self._schemes, C.POINTER(Scheme_t)),
                         C.cast(self._ptrs, C.POINTER(C.c_void_p)))
        tb = lib.mxmoe_block_table_bytes(C.byref(self.B))
        if tb == 0:
            raise MxmoeError(ERR_UNSUPPORTED, "mxmoe_block_table_bytes")
        host = (C.c_uint8 * tb)()
        _check(lib.mxmoe_block_table_fill(C.byref(self.B), host, tb), "mxmoe_block_table_fill")
        self.table = torch.frombuffer(bytearray(host), dtype=torch.uint8).to(device)
        self.T_max = T_max or cfg.T
        self.ws_bytes = lib.mxmoe_workspace_bytes(C.byref(self.B), self.T_max)
        self.ws = empty_aligned(self.ws_bytes, device)
        torch.cuda.synchronize()
        for ps in self.packed:
            for p in ps:
                p.release_sources()

    def workspace_layout(self, T: int) -> dict:
        lay = WsLayout_t()
        _check(load_library().mxmoe_workspace_layout(C.byref(self.B), T, C.byref(lay)), "mxmoe_workspace_layout")
        return {f: getattr(lay, f) for f in WS_FIELDS}

    def forward(self, x, topk_ids, topk_w, y=None, expert_mask: Optional[Sequence[int]] = None,
                skip_combine: bool = False, events=None, stream=None, router_logits=None,
                renormalize: bool = False, shared_logits=None, shared_w=None, fp32_slots: bool = False):
        """topk_ids / topk_w may be None when router_logits (fp32 [T,E]) is
        given; the router's choice is then left in the workspace.
        fp32_slots: keep the weighted down rows in fp32 (default: rounded to
        the activation dtype); slot_dtype() says which the last call used."""
        torch = _torch()
        lib = load_library()
        T = x.shape[0]
        if T > self.T_max:
            raise ValueError(f"T={T} exceeds the workspace sized for {self.T_max} tokens")
        if y is None:
            y = torch.empty_like(x)
        opts = None
        self._fp32_slots = bool(fp32_slots)
        if (expert_mask is not None or skip_combine or events is not None or router_logits is not None
                or shared_w is not None or fp32_slots):
            o = ForwardOpts_t()
            o.fp32_slots = 1 if fp32_slots else 0
            o.router_logits = _ptr(router_logits)
            o.renormalize = 1 if renormalize else 0
            o.shared_logits = _ptr(shared_logits)
            o.shared_w = _ptr(shared_w)
            if events is not None:
                o.events = events.array
            if expert_mask is not None:
                self._mask = (C.c_uint8 * len(expert_mask))(*[1 if v else 0 for v in expert_mask])
                o.expert_mask = C.cast(self._mask, C.POINTER(C.c_uint8))
            o.skip_combine = 1 if skip_combine else 0
            opts = C.byref(o)
        st = lib.mxmoe_moe_forward_ex(C.byref(self.B), _ptr(self.table), T, _ptr(x), _ptr(topk_ids), _ptr(topk_w),
                                      _ptr(y), _ptr(self.ws), self.ws_bytes, opts, _stream_ptr(stream))
        _check(st, "mxmoe_moe_forward")
        return y

    def forward_noalloc(self, x, topk_ids, topk_w, y=None, stream=None):
        """The forward through mxmoe_moe_forward_noalloc (the library's own
        scratch array instead of this block's workspace)."""
        torch = _torch()
        lib = load_library()
        if y is None:
            y = torch.empty_like(x)
        st = lib.mxmoe_moe_forward_noalloc(C.byref(self.B), _ptr(self.table), x.shape[0], _ptr(x), _ptr(topk_ids),
                                           _ptr(topk_w), _ptr(y), _stream_ptr(stream))
        _check(st, "mxmoe_moe_forward_noalloc")
        return y

    def slot_dtype(self):
        """torch dtype of the slot rows the last forward wrote."""
        torch = _torch()
        if getattr(self, "_fp32_slots", False):
            return torch.float32
        return torch.bfloat16 if self.act == "bf16" else torch.float16

    def slot_rows(self, T: int):
        """The last forward's weighted down rows [T, k + n_shared, H] as a
        float32 numpy array (exact: a 16-bit slot widens without rounding)."""
        cfg = self.cfg
        n = T * (cfg.k + cfg.n_shared) * cfg.H
        v = self.ws_view("slots", self.slot_dtype(), n, T)
        return v.float().cpu().numpy().reshape(T, cfg.k + cfg.n_shared, cfg.H)

    def ws_view(self, field: str, dtype, count: int, T: int):
        """Typed view of an intermediate buffer inside the workspace (after a forward)."""
        off = self.workspace_layout(T)[field]
        if off == (1 << 64) - 1:
            return None
        torch = _torch()
        nbytes = count * torch.empty((), dtype=dtype).element_size()
        return self.ws[off: off + nbytes].view(dtype)


# --------------------------------------------------------------- HIP events
class PhaseEvents:
    """2 * N_PHASES hipEvents for MoEBlock.forward(events=...), via the HIP runtime."""

    def __init__(self):
        self.hip = C.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [C.POINTER(C.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [C.c_void_p]
        self.hip.hipEventDestroy.argtypes = [C.c_void_p]
        self.array = (C.c_void_p * (2 * N_PHASES))()
        for i in range(2 * N_PHASES):
            ev = C.c_void_p()
            if self.hip.hipEventCreate(C.byref(ev)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.array[i] = ev
        self.array = C.cast(self.array, C.POINTER(C.c_void_p))

    def elapsed_ms(self):
        """Per-phase durations (ms) of the last forward recorded with these events."""
        out = []
        self.hip.hipEventSynchronize(self.array[2 * N_PHASES - 1])
        for i in range(N_PHASES):
            t = C.c_float()
            if self.hip.hipEventElapsedTime(C.byref(t), self.array[2 * i], self.array[2 * i + 1]) != 0:
                raise RuntimeError("hipEventElapsedTime failed")
            out.append(float(t.value))
        return out

    def span_ms(self):
        """Duration (ms) of the whole last forward recorded with these events."""
        self.hip.hipEventSynchronize(self.array[2 * N_PHASES - 1])
        t = C.c_float()
        if self.hip.hipEventElapsedTime(C.byref(t), self.array[0], self.array[2 * N_PHASES - 1]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(t.value)

    def __del__(self):
        try:
            for i in range(2 * N_PHASES):
                self.hip.hipEventDestroy(self.array[i])
        except Exception:
            pass
