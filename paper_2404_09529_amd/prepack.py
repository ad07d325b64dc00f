"""Python binding of the C ABI in ``include/prepack.h`` (ctypes).

Argument marshalling only: every step of the packed prefill runs in the HIP
library.  PyTorch provides device memory and streams.  The functions keep the
C names: ``pp_pack``, ``pp_pack_padded``, ``pp_plan_bounds``,
``pp_prefill_workspace_size``, ``pp_prefill``, ``pp_last_error``,
``pp_version``.  A missing library raises ``LibraryMissing``; there is no
fallback of any kind.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libprepack.so")

PP_OK, PP_ERR_INVALID_ARG, PP_ERR_TOO_LONG, PP_ERR_BUFFER_TOO_SMALL, PP_ERR_UNSUPPORTED, PP_ERR_HIP = 0, -1, -2, -3, -4, -5
PP_F32, PP_BF16 = 0, 1
PP_EPI_STORE, PP_EPI_RESIDUAL, PP_EPI_SWIGLU = 0, 1, 2
PP_QTILE = 128
PP_MTILE = 256

_i32p = ctypes.POINTER(ctypes.c_int32)


class LibraryMissing(ImportError):
    pass


class PrepackError(RuntimeError):
    def __init__(self, code: int, where: str, message: str):
        super().__init__(f"{where} failed with status {code}: {message}")
        self.code = code


class PPPlan(ctypes.Structure):
    _fields_ = [("k", ctypes.c_int32), ("capacity", ctypes.c_int32), ("n_rows", ctypes.c_int32),
                ("max_len", ctypes.c_int32), ("total_len", ctypes.c_int32), ("n_qtiles", ctypes.c_int32),
                ("n_mtiles", ctypes.c_int32), ("slot_cap", ctypes.c_int64), ("qtile_cap", ctypes.c_int64),
                ("mtile_cap", ctypes.c_int64),
                ("row_seg_ptr", _i32p), ("seg_prompt", _i32p), ("seg_start", _i32p), ("seg_len", _i32p),
                ("prompt_kv_off", _i32p), ("slot_seg", _i32p), ("slot_pos", _i32p), ("slot_kv", _i32p),
                ("qtile_seg", _i32p), ("qtile_q0", _i32p), ("mtile_m0", _i32p)]


class PPConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("dtype", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_theta", ctypes.c_float)]


class PPWeights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("attn_norm", ctypes.POINTER(ctypes.c_void_p)), ("wqkv", ctypes.POINTER(ctypes.c_void_p)),
                ("wo", ctypes.POINTER(ctypes.c_void_p)), ("mlp_norm", ctypes.POINTER(ctypes.c_void_p)),
                ("w_gateup", ctypes.POINTER(ctypes.c_void_p)), ("w_down", ctypes.POINTER(ctypes.c_void_p))]


class PPDPlan(ctypes.Structure):
    _fields_ = [("k", ctypes.c_int32), ("capacity", ctypes.c_int32), ("n_rows", ctypes.c_int32),
                ("max_len", ctypes.c_int32), ("total_len", ctypes.c_int32), ("n_qtiles", ctypes.c_int32),
                ("n_mtiles", ctypes.c_int32),
                ("seg_prompt", ctypes.c_void_p), ("seg_start", ctypes.c_void_p), ("seg_len", ctypes.c_void_p),
                ("prompt_kv_off", ctypes.c_void_p), ("slot_seg", ctypes.c_void_p), ("slot_pos", ctypes.c_void_p),
                ("slot_kv", ctypes.c_void_p), ("qtile_seg", ctypes.c_void_p), ("qtile_q0", ctypes.c_void_p),
                ("mtile_m0", ctypes.c_void_p)]


class PPGenLayout(ctypes.Structure):
    _fields_ = [("k", ctypes.c_int32), ("n_new", ctypes.c_int32), ("padded", ctypes.c_int32),
                ("max_len", ctypes.c_int32), ("ctx_rows", ctypes.c_int64), ("gen_rows", ctypes.c_int64),
                ("ctx_off", _i32p), ("ctx_span", _i32p), ("ctx_valid", _i32p), ("pos0", _i32p), ("gen_off", _i32p)]


class PPGenDLayout(ctypes.Structure):
    _fields_ = [("k", ctypes.c_int32), ("n_new", ctypes.c_int32), ("padded", ctypes.c_int32),
                ("max_len", ctypes.c_int32), ("ctx_rows", ctypes.c_int64), ("gen_rows", ctypes.c_int64),
                ("ctx_off", ctypes.c_void_p), ("ctx_span", ctypes.c_void_p), ("ctx_valid", ctypes.c_void_p),
                ("pos0", ctypes.c_void_p), ("gen_off", ctypes.c_void_p)]


_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises LibraryMissing if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise LibraryMissing(f"{LIB_PATH} is missing: build it with `python -m paper_2404_09529_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.pp_last_error.restype = ctypes.c_char_p
        L.pp_version.restype = ctypes.c_char_p
        L.pp_plan_bounds.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64),
                                     ctypes.POINTER(ctypes.c_int64),
                                     ctypes.POINTER(ctypes.c_int64)]
        L.pp_pack.argtypes = [_i32p, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(PPPlan)]
        L.pp_pack_padded.argtypes = [_i32p, ctypes.c_int32, ctypes.POINTER(PPPlan)]
        L.pp_prefill_workspace_size.argtypes = [ctypes.POINTER(PPConfig), ctypes.POINTER(PPDPlan),
                                                ctypes.POINTER(ctypes.c_size_t)]
        L.pp_prefill.argtypes = [ctypes.POINTER(PPConfig), ctypes.POINTER(PPWeights), ctypes.POINTER(PPDPlan),
                                 ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        cfgp, dpp = ctypes.POINTER(PPConfig), ctypes.POINTER(PPDPlan)
        L.pp_embed.argtypes = [i32, vp, i32, i32, vp, dpp, vp, vp]
        L.pp_rmsnorm.argtypes = [i32, vp, vp, i32, i32, f32, vp, vp]
        L.pp_gemm.argtypes = [i32, i32, vp, i64, vp, i64, vp, i64, i32, i32, i32, dpp, vp]
        L.pp_rope.argtypes = [cfgp, dpp, vp, vp, vp]
        L.pp_kv_scatter.argtypes = [cfgp, dpp, vp, vp, vp, vp]
        L.pp_attention.argtypes = [cfgp, dpp, vp, i64, vp, vp, vp, vp]
        L.pp_qkv_projection.argtypes = [cfgp, dpp, vp, vp, vp, vp, vp, vp, vp]
        L.pp_final_norm_unpack.argtypes = [vp, vp, i32, f32, dpp, vp, vp]
        L.pp_first_token_workspace_size.argtypes = [cfgp, dpp, ctypes.POINTER(ctypes.c_size_t)]
        L.pp_first_token.argtypes = [cfgp, dpp, vp, vp, vp, ctypes.c_size_t, vp, vp, vp]
        L.pp_first_token_noalloc.argtypes = [cfgp, dpp, vp, vp, vp, vp, vp]
        glp, gdp, wp = ctypes.POINTER(PPGenLayout), ctypes.POINTER(PPGenDLayout), ctypes.POINTER(PPWeights)
        L.pp_gen_layout_make.argtypes = [_i32p, i32, i32, i32, glp]
        L.pp_decode_workspace_size.argtypes = [cfgp, gdp, ctypes.POINTER(ctypes.c_size_t)]
        L.pp_decode_step.argtypes = [cfgp, wp, gdp, i32, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp, vp, vp]
        L.pp_generate.argtypes = [cfgp, wp, gdp, i32, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp, vp]
        for name in ("pp_plan_bounds", "pp_pack", "pp_pack_padded", "pp_prefill_workspace_size", "pp_prefill",
                     "pp_embed", "pp_rmsnorm", "pp_gemm", "pp_rope", "pp_kv_scatter", "pp_attention",
                     "pp_final_norm_unpack", "pp_first_token_workspace_size", "pp_first_token",
                     "pp_first_token_noalloc",
                     "pp_gen_layout_make", "pp_decode_workspace_size", "pp_decode_step", "pp_generate"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def pp_last_error() -> str:
    return lib().pp_last_error().decode()


def pp_version() -> str:
    return lib().pp_version().decode()


def _check(status: int, where: str) -> None:
    if status != PP_OK:
        raise PrepackError(status, where, pp_last_error())


# ----------------------------------------------------------------------------- planning
@dataclass
class Plan:
    k: int
    capacity: int
    n_rows: int
    max_len: int
    total_len: int
    row_seg_ptr: np.ndarray
    seg_prompt: np.ndarray
    seg_start: np.ndarray
    seg_len: np.ndarray
    prompt_kv_off: np.ndarray
    slot_seg: np.ndarray
    slot_pos: np.ndarray
    slot_kv: np.ndarray
    qtile_seg: np.ndarray
    qtile_q0: np.ndarray
    mtile_m0: np.ndarray

    @property
    def n_slots(self) -> int:
        return self.n_rows * self.capacity

    @property
    def n_qtiles(self) -> int:
        return int(self.qtile_seg.size)

    @property
    def n_mtiles(self) -> int:
        return int(self.mtile_m0.size)


def pp_plan_bounds(k: int, C: int):
    """(slot_cap, qtile_cap, mtile_cap) of a plan of k prompts in rows of C slots."""
    s, q, m = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(lib().pp_plan_bounds(k, C, ctypes.byref(s), ctypes.byref(q), ctypes.byref(m)), "pp_plan_bounds")
    return s.value, q.value, m.value


_PLAN_ARRAYS = ("row_seg_ptr", "seg_prompt", "seg_start", "seg_len", "prompt_kv_off", "slot_seg", "slot_pos",
                "slot_kv", "qtile_seg", "qtile_q0", "mtile_m0")


def _plan_arrays(k: int, bs: int, bq: int, bm: int):
    sizes = {"row_seg_ptr": k + 1, "seg_prompt": k, "seg_start": k, "seg_len": k, "prompt_kv_off": k + 1,
             "slot_seg": bs, "slot_pos": bs, "slot_kv": bs, "qtile_seg": bq, "qtile_q0": bq, "mtile_m0": bm}
    return {n: np.empty(max(sizes[n], 1), dtype=np.int32) for n in _PLAN_ARRAYS}


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(_i32p)


def _run_pack(lengths: Sequence[int], capacity: Optional[int], slot_cap=None, qtile_cap=None,
              mtile_cap=None) -> Plan:
    L = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    k = int(L.size)
    m = int(L.max()) if k else 0
    C = m if (capacity is None or capacity == 0) else int(capacity)
    bs, bq, bm = pp_plan_bounds(k, max(C, 0)) if C >= 0 else (0, 0, 0)
    bs = bs if slot_cap is None else slot_cap
    bq = bq if qtile_cap is None else qtile_cap
    bm = bm if mtile_cap is None else mtile_cap
    arrs = _plan_arrays(k, bs, bq, bm)
    p = PPPlan(slot_cap=bs, qtile_cap=bq, mtile_cap=bm, **{n: _ptr(a) for n, a in arrs.items()})
    if capacity is None:
        _check(lib().pp_pack_padded(_ptr(L) if k else None, k, ctypes.byref(p)), "pp_pack_padded")
    else:
        _check(lib().pp_pack(_ptr(L) if k else None, k, int(capacity), ctypes.byref(p)), "pp_pack")
    T = p.n_rows * p.capacity
    return Plan(k=p.k, capacity=p.capacity, n_rows=p.n_rows, max_len=p.max_len, total_len=p.total_len,
                row_seg_ptr=arrs["row_seg_ptr"][: p.n_rows + 1].copy(), seg_prompt=arrs["seg_prompt"][:k].copy(),
                seg_start=arrs["seg_start"][:k].copy(), seg_len=arrs["seg_len"][:k].copy(),
                prompt_kv_off=arrs["prompt_kv_off"][: k + 1].copy(), slot_seg=arrs["slot_seg"][:T].copy(),
                slot_pos=arrs["slot_pos"][:T].copy(), slot_kv=arrs["slot_kv"][:T].copy(),
                qtile_seg=arrs["qtile_seg"][: p.n_qtiles].copy(), qtile_q0=arrs["qtile_q0"][: p.n_qtiles].copy(),
                mtile_m0=arrs["mtile_m0"][: p.n_mtiles].copy())


class PlanBuffers:
    """Host arrays for plans of up to k prompts in rows of up to C slots, allocated once, so
    that packing batch after batch costs only the C call (``pack`` returns the filled pp_plan
    struct; its arrays stay valid until the next call)."""

    def __init__(self, k: int, C: int):
        bs, bq, bm = pp_plan_bounds(k, C)
        self.k = k
        self.arrs = _plan_arrays(k, bs, bq, bm)
        self.struct = PPPlan(slot_cap=bs, qtile_cap=bq, mtile_cap=bm, **{n: _ptr(a) for n, a in self.arrs.items()})

    def pack(self, lengths: np.ndarray, capacity: int) -> PPPlan:
        """pp_pack of int32 contiguous ``lengths`` (at most k of them, rows of at most C)."""
        _check(lib().pp_pack(_ptr(lengths), int(lengths.size), int(capacity), ctypes.byref(self.struct)),
               "pp_pack")
        return self.struct


def pp_pack(lengths: Sequence[int], capacity: int = 0, **caps) -> Plan:
    """First-fit-decreasing packing into rows of ``capacity`` slots (0 = max length)."""
    return _run_pack(lengths, capacity, **caps)


def pp_pack_padded(lengths: Sequence[int], **caps) -> Plan:
    """Full-batching plan: one right-padded row of length max(lengths) per prompt."""
    return _run_pack(lengths, None, **caps)


# ----------------------------------------------------------------------------- device side
def _torch():
    import torch
    return torch


class DevicePlan:
    """A plan's arrays in device memory plus the pp_dplan struct that points at them."""

    def __init__(self, plan: Plan, device="cuda"):
        torch = _torch()
        self.plan = plan
        self.tensors = {n: torch.from_numpy(np.ascontiguousarray(getattr(plan, n))).to(device)
                        for n in ("seg_prompt", "seg_start", "seg_len", "prompt_kv_off", "slot_seg", "slot_pos",
                                  "slot_kv", "qtile_seg", "qtile_q0", "mtile_m0")}
        self.struct = PPDPlan(k=plan.k, capacity=plan.capacity, n_rows=plan.n_rows, max_len=plan.max_len,
                              total_len=plan.total_len, n_qtiles=plan.n_qtiles, n_mtiles=plan.n_mtiles,
                              **{n: t.data_ptr() for n, t in self.tensors.items()})


def interleave_gate_up(wg, wu):
    """[F, d] x2 -> [2F, d] with rows 32j..32j+15 = wg[16j..16j+15], 32j+16..32j+31 = wu[16j..]."""
    F, d = wg.shape
    assert F % 16 == 0
    return _torch().stack([wg.reshape(F // 16, 16, d), wu.reshape(F // 16, 16, d)], dim=1).reshape(2 * F, d)


class DeviceModel:
    """Decoder weights on the device in the library's layout, plus pp_config / pp_weights."""

    def __init__(self, shape, weights: Dict, device="cuda"):
        torch = _torch()
        self.shape = shape
        dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        self.dtype_code = PP_BF16 if shape.dtype == "bf16" else PP_F32
        self.torch_dtype = dt

        def dev(a, t=dt):
            if isinstance(a, torch.Tensor):          # already drawn with torch (device or host)
                return a.to(device=device, dtype=t)
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device=device).to(t)

        self.embed = dev(weights["embed"])
        self.final_norm = dev(weights["final_norm"], torch.float32)
        self.layers: List[Dict] = []
        for L in weights["layers"][: shape.n_layers]:
            wqkv = torch.cat([dev(L["wq"]), dev(L["wk"]), dev(L["wv"])], dim=0)
            self.layers.append(dict(
                attn_norm=dev(L["attn_norm"], torch.float32), wqkv=wqkv, wo=dev(L["wo"]),
                mlp_norm=dev(L["mlp_norm"], torch.float32),
                w_gateup=interleave_gate_up(dev(L["wg"]), dev(L["wu"])).contiguous(), w_down=dev(L["wd"])))
        n = shape.n_layers
        self._arrays = {key: (ctypes.c_void_p * n)(*[Ld[key].data_ptr() for Ld in self.layers])
                        for key in ("attn_norm", "wqkv", "wo", "mlp_norm", "w_gateup", "w_down")}
        vp = ctypes.POINTER(ctypes.c_void_p)
        self.weights_struct = PPWeights(embed=self.embed.data_ptr(), final_norm=self.final_norm.data_ptr(),
                                        **{k: ctypes.cast(a, vp) for k, a in self._arrays.items()})
        self.config = PPConfig(n_layers=n, d_model=shape.d_model, n_heads=shape.n_heads,
                               n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim, ffn_dim=shape.ffn_dim,
                               vocab=shape.vocab, dtype=self.dtype_code, rms_eps=shape.rms_eps,
                               rope_theta=shape.rope_theta)


def pp_prefill_workspace_size(model: DeviceModel, dplan: DevicePlan) -> int:
    n = ctypes.c_size_t()
    _check(lib().pp_prefill_workspace_size(ctypes.byref(model.config), ctypes.byref(dplan.struct),
                                           ctypes.byref(n)), "pp_prefill_workspace_size")
    return n.value


def pp_prefill(model: DeviceModel, dplan: DevicePlan, tokens, workspace, hidden, k_cache, v_cache,
               stream=None) -> None:
    """Enqueue the packed prefill on ``stream`` (default: torch's current stream)."""
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    _check(lib().pp_prefill(ctypes.byref(model.config), ctypes.byref(model.weights_struct),
                            ctypes.byref(dplan.struct), tokens.data_ptr(), workspace.data_ptr(),
                            workspace.numel() * workspace.element_size(), hidden.data_ptr(),
                            k_cache.data_ptr(), v_cache.data_ptr(), ctypes.c_void_p(stream.cuda_stream)),
           "pp_prefill")


class Prefill:
    """Outputs and workspace for one (model, plan) pair, allocated once with torch."""

    def __init__(self, model: DeviceModel, dplan: DevicePlan, device="cuda"):
        torch = _torch()
        s = model.shape
        L = dplan.plan.total_len
        self.model, self.dplan = model, dplan
        self.workspace = torch.empty(max(pp_prefill_workspace_size(model, dplan), 1), dtype=torch.uint8,
                                     device=device)
        self.hidden = torch.empty((L, s.d_model), dtype=torch.float32, device=device)
        kv = (s.n_layers, L, s.n_kv_heads * s.head_dim)
        self.k_cache = torch.empty(kv, dtype=model.torch_dtype, device=device)
        self.v_cache = torch.empty(kv, dtype=model.torch_dtype, device=device)

    def __call__(self, tokens, stream=None):
        pp_prefill(self.model, self.dplan, tokens, self.workspace, self.hidden, self.k_cache, self.v_cache, stream)
        return self.hidden, self.k_cache, self.v_cache


# ----------------------------------------------------------------------------- single steps
def config_of(shape, n_layers: Optional[int] = None) -> PPConfig:
    return PPConfig(n_layers=shape.n_layers if n_layers is None else n_layers, d_model=shape.d_model,
                    n_heads=shape.n_heads, n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                    ffn_dim=shape.ffn_dim, vocab=shape.vocab,
                    dtype=PP_BF16 if shape.dtype == "bf16" else PP_F32, rms_eps=shape.rms_eps,
                    rope_theta=shape.rope_theta)


def _stream(stream):
    if stream is None:
        stream = _torch().cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _p(t):
    return None if t is None else t.data_ptr()


def pp_embed(dtype: int, embed, vocab: int, d: int, tokens, dplan: DevicePlan, x, stream=None) -> None:
    _check(lib().pp_embed(dtype, _p(embed), vocab, d, _p(tokens), ctypes.byref(dplan.struct), _p(x),
                          _stream(stream)), "pp_embed")


def pp_rmsnorm(dtype: int, x, gain, rows: int, d: int, eps: float, out, stream=None) -> None:
    _check(lib().pp_rmsnorm(dtype, _p(x), _p(gain), rows, d, eps, _p(out), _stream(stream)), "pp_rmsnorm")


def pp_gemm(dtype: int, epilogue: int, A, lda: int, B, ldb: int, C, ldc: int, M: int, N: int, K: int,
            dplan: Optional[DevicePlan] = None, stream=None) -> None:
    _check(lib().pp_gemm(dtype, epilogue, _p(A), lda, _p(B), ldb, _p(C), ldc, M, N, K,
                         None if dplan is None else ctypes.byref(dplan.struct), _stream(stream)), "pp_gemm")


def pp_rope(cfg: PPConfig, dplan: DevicePlan, qkv, table, stream=None) -> None:
    _check(lib().pp_rope(ctypes.byref(cfg), ctypes.byref(dplan.struct), _p(qkv), _p(table), _stream(stream)),
           "pp_rope")


def pp_kv_scatter(cfg: PPConfig, dplan: DevicePlan, qkv, k_cache, v_cache, stream=None) -> None:
    _check(lib().pp_kv_scatter(ctypes.byref(cfg), ctypes.byref(dplan.struct), _p(qkv), _p(k_cache), _p(v_cache),
                               _stream(stream)), "pp_kv_scatter")


def pp_qkv_projection(cfg: PPConfig, dplan: DevicePlan, xn, wqkv, table, q_out, k_cache, v_cache,
                      stream=None) -> None:
    _check(lib().pp_qkv_projection(ctypes.byref(cfg), ctypes.byref(dplan.struct), _p(xn), _p(wqkv), _p(table),
                                   _p(q_out), _p(k_cache), _p(v_cache), _stream(stream)), "pp_qkv_projection")


def pp_attention(cfg: PPConfig, dplan: DevicePlan, q, ldq: int, k_cache, v_cache, out, stream=None) -> None:
    _check(lib().pp_attention(ctypes.byref(cfg), ctypes.byref(dplan.struct), _p(q), ldq, _p(k_cache),
                              _p(v_cache), _p(out), _stream(stream)), "pp_attention")


def pp_final_norm_unpack(x, gain, d: int, eps: float, dplan: DevicePlan, hidden, stream=None) -> None:
    _check(lib().pp_final_norm_unpack(_p(x), _p(gain), d, eps, ctypes.byref(dplan.struct), _p(hidden),
                                      _stream(stream)), "pp_final_norm_unpack")


def pp_first_token_workspace_size(cfg: PPConfig, dplan: DevicePlan) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().pp_first_token_workspace_size(ctypes.byref(cfg), ctypes.byref(dplan.struct), ctypes.byref(n)),
           "pp_first_token_workspace_size")
    return n.value


def pp_first_token(cfg: PPConfig, dplan: DevicePlan, hidden, lm_head, workspace, tokens, logits=None,
                   stream=None) -> None:
    """Greedy first token of every prompt: tokens [k] int32 (and logits [k, vocab] float32)."""
    _check(lib().pp_first_token(ctypes.byref(cfg), ctypes.byref(dplan.struct), _p(hidden), _p(lm_head),
                                _p(workspace), workspace.numel() * workspace.element_size(), _p(logits),
                                _p(tokens), _stream(stream)), "pp_first_token")



PP_FIRST_TOKEN_SCRATCH_BYTES = 16 << 20


def pp_first_token_noalloc(cfg: PPConfig, dplan: DevicePlan, hidden, lm_head, tokens, logits=None,
                           stream=None) -> None:
    """pp_first_token with the library's static device workspace (allocates nothing)."""
    _check(lib().pp_first_token_noalloc(ctypes.byref(cfg), ctypes.byref(dplan.struct), _p(hidden), _p(lm_head),
                                        _p(logits), _p(tokens), _stream(stream)), "pp_first_token_noalloc")


# ----------------------------------------------------------------------------- generation
@dataclass
class GenLayout:
    """Host copy of a pp_gen_layout: where each prompt's keys and values live while generating."""
    k: int
    n_new: int
    padded: bool
    max_len: int
    ctx_rows: int
    gen_rows: int
    ctx_off: np.ndarray
    ctx_span: np.ndarray
    ctx_valid: np.ndarray
    pos0: np.ndarray
    gen_off: np.ndarray


_GEN_ARRAYS = ("ctx_off", "ctx_span", "ctx_valid", "pos0", "gen_off")


def pp_gen_layout_make(lengths: Sequence[int], n_new: int, padded: bool = False) -> GenLayout:
    """Cache layout for generating n_new tokens per prompt: packed, or full batching."""
    L = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    k = int(L.size)
    arrs = {n: np.zeros(max(k, 1), dtype=np.int32) for n in _GEN_ARRAYS}
    g = PPGenLayout(**{n: _ptr(a) for n, a in arrs.items()})
    _check(lib().pp_gen_layout_make(_ptr(L) if k else None, k, int(n_new), int(bool(padded)), ctypes.byref(g)),
           "pp_gen_layout_make")
    return GenLayout(k=g.k, n_new=g.n_new, padded=bool(g.padded), max_len=g.max_len, ctx_rows=g.ctx_rows,
                     gen_rows=g.gen_rows, **{n: a[:k].copy() for n, a in arrs.items()})


class DeviceGenLayout:
    """A generation layout's arrays in device memory plus the pp_gen_dlayout struct."""

    def __init__(self, layout: GenLayout, device="cuda"):
        torch = _torch()
        self.layout = layout
        self.tensors = {n: torch.from_numpy(getattr(layout, n)).to(device) for n in _GEN_ARRAYS}
        self.struct = PPGenDLayout(k=layout.k, n_new=layout.n_new, padded=int(layout.padded),
                                   max_len=layout.max_len, ctx_rows=layout.ctx_rows, gen_rows=layout.gen_rows,
                                   **{n: t.data_ptr() for n, t in self.tensors.items()})


def pp_decode_workspace_size(model: DeviceModel, dlayout: DeviceGenLayout) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().pp_decode_workspace_size(ctypes.byref(model.config), ctypes.byref(dlayout.struct),
                                          ctypes.byref(n)), "pp_decode_workspace_size")
    return n.value


def pp_decode_step(model: DeviceModel, dlayout: DeviceGenLayout, step: int, tokens_in, lm_head, ctx_k, ctx_v,
                   gen_k, gen_v, workspace, tokens_out, logits=None, stream=None) -> None:
    """One greedy decode step of every prompt (see pp_decode_step in include/prepack.h)."""
    _check(lib().pp_decode_step(ctypes.byref(model.config), ctypes.byref(model.weights_struct),
                                ctypes.byref(dlayout.struct), int(step), _p(tokens_in), _p(lm_head), _p(ctx_k),
                                _p(ctx_v), _p(gen_k), _p(gen_v), _p(workspace),
                                workspace.numel() * workspace.element_size(), _p(logits), _p(tokens_out),
                                _stream(stream)), "pp_decode_step")


def pp_generate(model: DeviceModel, dlayout: DeviceGenLayout, n_steps: int, tokens_first, lm_head, ctx_k, ctx_v,
                gen_k, gen_v, workspace, tokens, stream=None) -> None:
    """n_steps greedy decode steps back to back: tokens [n_steps, k] int32."""
    _check(lib().pp_generate(ctypes.byref(model.config), ctypes.byref(model.weights_struct),
                             ctypes.byref(dlayout.struct), int(n_steps), _p(tokens_first), _p(lm_head), _p(ctx_k),
                             _p(ctx_v), _p(gen_k), _p(gen_v), _p(workspace),
                             workspace.numel() * workspace.element_size(), _p(tokens), _stream(stream)),
           "pp_generate")


class Generation:
    """Caches and workspace for greedy generation after a prefill (allocated once with torch).

    packed: the prefill's per-prompt caches are the context; the generated keys and values go
    to a cache of n_new rows per prompt.  padded (full batching): one cache of k rows of
    m + n_new slots, into which the prefill's caches are placed once at set-up (a copy that
    is part of building the baseline's layout, not of its decode steps)."""

    def __init__(self, model: DeviceModel, prefill: "Prefill", lengths: Sequence[int], n_new: int,
                 padded: bool = False, device="cuda"):
        torch = _torch()
        s = model.shape
        self.model, self.n_new, self.padded = model, int(n_new), bool(padded)
        self.layout = pp_gen_layout_make(lengths, n_new, padded)
        self.dlayout = DeviceGenLayout(self.layout, device)
        kvw = s.n_kv_heads * s.head_dim
        rows = (s.n_layers, self.layout.gen_rows, kvw)
        if padded:
            self.gen_k = torch.zeros(rows, dtype=model.torch_dtype, device=device)
            self.gen_v = torch.zeros(rows, dtype=model.torch_dtype, device=device)
            lay = self.layout
            dest = np.concatenate([lay.ctx_off[i] + np.arange(lay.ctx_valid[i]) for i in range(lay.k)])
            idx = torch.from_numpy(dest.astype(np.int64)).to(device)
            self.gen_k.index_copy_(1, idx, prefill.k_cache)
            self.gen_v.index_copy_(1, idx, prefill.v_cache)
            self.ctx_k, self.ctx_v = self.gen_k, self.gen_v
        else:
            self.ctx_k, self.ctx_v = prefill.k_cache, prefill.v_cache
            self.gen_k = torch.empty(rows, dtype=model.torch_dtype, device=device)
            self.gen_v = torch.empty(rows, dtype=model.torch_dtype, device=device)
        self.workspace = torch.empty(max(pp_decode_workspace_size(model, self.dlayout), 1), dtype=torch.uint8,
                                     device=device)
        self.tokens = torch.empty((self.n_new, self.layout.k), dtype=torch.int32, device=device)

    def kv_cache_bytes(self) -> int:
        """Bytes of key/value cache this layout holds for the whole generation."""
        t = [self.gen_k, self.gen_v] + ([] if self.padded else [self.ctx_k, self.ctx_v])
        return int(sum(x.numel() * x.element_size() for x in t))

    def step(self, step: int, tokens_in, lm_head, tokens_out, logits=None, stream=None) -> None:
        pp_decode_step(self.model, self.dlayout, step, tokens_in, lm_head, self.ctx_k, self.ctx_v, self.gen_k,
                       self.gen_v, self.workspace, tokens_out, logits, stream)

    def __call__(self, tokens_first, lm_head, n_steps: Optional[int] = None, stream=None):
        n = self.n_new if n_steps is None else n_steps
        pp_generate(self.model, self.dlayout, n, tokens_first, lm_head, self.ctx_k, self.ctx_v, self.gen_k,
                    self.gen_v, self.workspace, self.tokens, stream)
        return self.tokens[:n]

    def capture(self, tokens_first, lm_head, n_steps: Optional[int] = None):
        """Record the whole pp_generate call (every launch of every step) into a HIP graph
        with torch's graph capture; replay() then re-runs it with one launch from the host.
        The graph is bound to these buffers, tokens_first and lm_head included: refill
        tokens_first in place before a replay to generate from new first tokens."""
        torch = _torch()
        n = self.n_new if n_steps is None else n_steps
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):             # warm-up off the capture, as torch requires
            self(tokens_first, lm_head, n)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self(tokens_first, lm_head, n)
        return self.tokens[:n]

    def replay(self):
        self.graph.replay()
        return self.tokens
