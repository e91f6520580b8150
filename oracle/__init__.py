"""CPU oracle for the Prox sparse SwiGLU FFN decode step.

TEST INFRASTRUCTURE ONLY.  The oracle is the plain fp64 reference that the
HIP path is checked against.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it; the product package never does.

The arithmetic lives in ``oracle.c`` (plain C, binary64, no FMA contraction);
this module only builds it with gcc and marshals numpy arrays through ctypes.
Each wrapper names the passage of the paper its C function follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

PROXY_QUANT = 0   # W~ from codes/scales
PROXY_NONE = 1    # W~ = W (unquantised proxy)
SILU, GELU = 0, 1  # gate activation: SwiGLU (Sec. 2.1) or GeGLU


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` with gcc (OpenMP, -O2)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
               "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        L = ctypes.CDLL(_LIB)
        P, I, D = ctypes.c_void_p, ctypes.c_int, ctypes.c_double
        L.oracle_half_to_double.argtypes = [ctypes.c_uint16, I]
        L.oracle_half_to_double.restype = D
        L.oracle_double_to_f16.argtypes = [D]
        L.oracle_double_to_f16.restype = ctypes.c_uint16
        L.oracle_quantize.argtypes = [P, I, I, I, I, I, P, P]
        L.oracle_topk.argtypes = [P, I, I, P]
        L.oracle_select_inputs.argtypes = [P, I, I, I, I, P]
        L.oracle_proxy.argtypes = [P, I, I, I, I, P, I, I, P, P, P, P, I, P, P, P, P, P, P, I]
        L.oracle_select_channels.argtypes = [P, I, I, P]
        L.oracle_stage2.argtypes = [P, I, I, I, I, P, P, P, P, I, P, P, I]
        L.oracle_ffn_dense.argtypes = [P, I, I, I, I, P, P, P, P, I]
        L.oracle_stage2_w4.argtypes = [P, I, I, I, I, P, P, P, P, P, P, P, I, P, P, I]
        L.oracle_ffn_sparse.argtypes = [P, I, I, I, I, P, P, P, I, P, P, P, P, I, I, I,
                                        P, P, P, P, P, I]
        L.oracle_add_rmsnorm.argtypes = [P, P, I, I, I, D, P]
        L.oracle_double_to_bf16.argtypes = [D]
        L.oracle_double_to_bf16.restype = ctypes.c_uint16
        L.oracle_round_to_dtype.argtypes = [P, I, I, P]
        L.oracle_halves_to_double.argtypes = [P, I, I, P]
        L.oracle_select_threshold.argtypes = [P, I, D, P]
        L.oracle_select_threshold.restype = I
        L.oracle_select_inputs_tau.argtypes = [P, I, I, I, D, P]
        L.oracle_select_inputs_tau.restype = I
        L.oracle_ffn_sparse_tau.argtypes = [P, I, I, I, I, P, P, P, I, P, P, P, P, I, D, D,
                                            P, I, P, P, P, P, P, I]
        L.oracle_gate_act.argtypes = [D, I]
        L.oracle_gate_act.restype = D
        L.oracle_reservoir_add.argtypes = [P, I, P, P, I, P]
        L.oracle_quantile_threshold.argtypes = [P, I, D]
        L.oracle_quantile_threshold.restype = D
        L.oracle_prox_cost.argtypes = [D, D, D]
        L.oracle_prox_cost.restype = D
        L.oracle_effective_sparsity.argtypes = [D, D, D]
        L.oracle_effective_sparsity.restype = D
        L.oracle_allocate.argtypes = [D, D, D, D, D, P, P]
        L.oracle_max_threads.restype = I
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _u16(a):
    return np.ascontiguousarray(a, dtype=np.uint16)


def half_to_double(bits: int, dtype: int) -> float:
    return lib().oracle_half_to_double(int(bits), int(dtype))


def double_to_f16(v: float) -> int:
    """IEEE binary16 round-to-nearest-even of a double (bit pattern)."""
    return int(lib().oracle_double_to_f16(float(v)))


def quantize(w, dtype: int, bits: int, group: int):
    """Sec. 4.3 symmetric proxy quantisation of a channel-major [f][d] matrix.
    Returns (codes int8 [f][d], scales fp16-bits uint16 [f][d/group])."""
    w = _u16(w)
    f, d = w.shape
    assert d % group == 0
    codes = np.empty((f, d), np.int8)
    scales = np.empty((f, d // group), np.uint16)
    lib().oracle_quantize(_p(w), dtype, d, f, bits, group, _p(codes), _p(scales))
    return codes, scales


def topk(key, k: int):
    """App. A.6 top-k: ascending indices of the k largest keys, ties to the lower index."""
    key = np.ascontiguousarray(key, dtype=np.float64)
    out = np.empty(k, np.int32)
    lib().oracle_topk(_p(key), key.size, k, _p(out))
    return out


def select_inputs(x, dtype: int, k_in: int):
    """Sec. 4.1 input mask as top-k over a_i = max_b |x_{b,i}|; x is [B][d]."""
    x = _u16(np.atleast_2d(x))
    B, d = x.shape
    out = np.empty(k_in, np.int32)
    lib().oracle_select_inputs(_p(x), dtype, B, d, k_in, _p(out))
    return out


def proxy(x, dtype: int, in_idx, *, codes_g=None, scales_g=None, codes_u=None,
          scales_u=None, group: int = 0, w_gate=None, w_up=None, kind=PROXY_QUANT, act=SILU):
    """Sec. 4.1 Stage 1: returns (g~ [B][f], u~ [B][f], s~ [B][f], score [f])."""
    x = _u16(np.atleast_2d(x))
    B, d = x.shape
    in_idx = np.ascontiguousarray(in_idx, dtype=np.int32)
    if kind == PROXY_QUANT:
        codes_g = np.ascontiguousarray(codes_g, np.int8)
        codes_u = np.ascontiguousarray(codes_u, np.int8)
        scales_g, scales_u = _u16(scales_g), _u16(scales_u)
        f = codes_g.shape[0]
    else:
        w_gate, w_up = _u16(w_gate), _u16(w_up)
        f = w_gate.shape[0]
    gt = np.empty((B, f)); ut = np.empty((B, f)); st = np.empty((B, f)); sc = np.empty(f)
    lib().oracle_proxy(_p(x), dtype, B, d, f, _p(in_idx), in_idx.size, kind,
                       _p(codes_g), _p(scales_g), _p(codes_u), _p(scales_u), group,
                       _p(w_gate), _p(w_up), _p(gt), _p(ut), _p(st), _p(sc), act)
    return gt, ut, st, sc


def select_channels(score, k_ff: int):
    """Sec. 4.1 channel mask as top-k over the proxy score."""
    return topk(score, k_ff)


def stage2(x, dtype: int, w_gate, w_up, w_down, ff_idx, act=SILU):
    """Sec. 4.1 Stage 2 on channels ff_idx: returns (s [B][k_ff], y [B][d])."""
    x = _u16(np.atleast_2d(x))
    B, d = x.shape
    wg, wu, wd = _u16(w_gate), _u16(w_up), _u16(w_down)
    f = wg.shape[0]
    ff_idx = np.ascontiguousarray(ff_idx, dtype=np.int32)
    s = np.empty((B, max(ff_idx.size, 1)))
    y = np.empty((B, d))
    lib().oracle_stage2(_p(x), dtype, B, d, f, _p(wg), _p(wu), _p(wd), _p(ff_idx),
                        ff_idx.size, _p(s), _p(y), act)
    return s[:, :ff_idx.size], y


def stage2_w4(x, dtype: int, w4, ff_idx, act=SILU):
    """Stage 2 on INT4 base weights (W4A16; Sec. 5.1 names the combination
    as future work).  w4 = dict(codes_g, scales_g, codes_u, scales_u, codes_d,
    scales_d, group): each matrix as quantize(w, dtype, 4, group) returns it.
    Returns (s [B][k_ff], y [B][d]) in fp64."""
    x = _u16(np.atleast_2d(x))
    B, d = x.shape
    c = {k: np.ascontiguousarray(w4[k], np.int8) for k in ("codes_g", "codes_u", "codes_d")}
    sc = {k: _u16(w4[k]) for k in ("scales_g", "scales_u", "scales_d")}
    ff_idx = np.ascontiguousarray(ff_idx, dtype=np.int32)
    s = np.empty((B, max(ff_idx.size, 1)))
    y = np.empty((B, d))
    lib().oracle_stage2_w4(_p(x), dtype, B, d, int(w4["group"]), _p(c["codes_g"]),
                           _p(sc["scales_g"]), _p(c["codes_u"]), _p(sc["scales_u"]),
                           _p(c["codes_d"]), _p(sc["scales_d"]), _p(ff_idx), ff_idx.size,
                           _p(s), _p(y), act)
    return s[:, :ff_idx.size], y


def quantize_w4(w_gate, w_up, w_down, dtype: int, group: int) -> dict:
    """The three base matrices in the 4-bit group format stage2_w4 takes."""
    out = {"group": group}
    for key, w in (("g", w_gate), ("u", w_up), ("d", w_down)):
        out["codes_" + key], out["scales_" + key] = quantize(w, dtype, 4, group)
    return out


def ffn_dense_w4(x, dtype: int, w4, act=SILU):
    """The dense FFN on INT4 base weights: stage2_w4 over every channel."""
    f = np.asarray(w4["codes_g"]).shape[0]
    return stage2_w4(x, dtype, w4, np.arange(f, dtype=np.int32), act)[1]


def ffn_sparse_w4(x, dtype: int, w4, k_in: int, k_ff: int, *, codes_g, scales_g, codes_u,
                  scales_u, group: int, act=SILU):
    """The Sec. 4.1 decode step with Stage 2 on INT4 base weights: input
    top-k, the INT4 proxy score, channel top-k, then stage2_w4.  The proxy
    arguments are those of proxy() (a proxy of the original weights).
    Returns dict(y, in_idx, score, ff_idx)."""
    in_idx = select_inputs(x, dtype, k_in)
    _, _, _, score = proxy(x, dtype, in_idx, codes_g=codes_g, scales_g=scales_g,
                           codes_u=codes_u, scales_u=scales_u, group=group, act=act)
    ff_idx = select_channels(score, k_ff)
    _, y = stage2_w4(x, dtype, w4, ff_idx, act)
    return {"y": y, "in_idx": in_idx, "score": score, "ff_idx": ff_idx}


def ffn_dense(x, dtype: int, w_gate, w_up, w_down, act=SILU):
    """Sec. 2.1 dense SwiGLU FFN in fp64: y [B][d]."""
    x = _u16(np.atleast_2d(x))
    B, d = x.shape
    wg, wu, wd = _u16(w_gate), _u16(w_up), _u16(w_down)
    y = np.empty((B, d))
    lib().oracle_ffn_dense(_p(x), dtype, B, d, wg.shape[0], _p(wg), _p(wu), _p(wd), _p(y), act)
    return y


def ffn_sparse(x, dtype: int, w_gate, w_up, w_down, k_in: int, k_ff: int, *,
               codes_g=None, scales_g=None, codes_u=None, scales_u=None, group: int = 0,
               kind=PROXY_QUANT, mask_override=None, act=SILU):
    """Whole Sec. 4.1 decode step.  Returns dict(y, in_idx, score, ff_idx)."""
    x = _u16(np.atleast_2d(x))
    B, d = x.shape
    wg, wu, wd = _u16(w_gate), _u16(w_up), _u16(w_down)
    f = wg.shape[0]
    if kind == PROXY_QUANT:
        codes_g = np.ascontiguousarray(codes_g, np.int8)
        codes_u = np.ascontiguousarray(codes_u, np.int8)
        scales_g, scales_u = _u16(scales_g), _u16(scales_u)
    mo = None if mask_override is None else np.ascontiguousarray(mask_override, np.int32)
    if mo is not None:
        assert mo.size == k_ff
    in_idx = np.empty(k_in, np.int32)
    score = np.empty(f)
    ff_idx = np.empty(k_ff, np.int32)
    y = np.empty((B, d))
    lib().oracle_ffn_sparse(_p(x), dtype, B, d, f, _p(wg), _p(wu), _p(wd), kind,
                            _p(codes_g), _p(scales_g), _p(codes_u), _p(scales_u), group,
                            k_in, k_ff, _p(mo), _p(in_idx), _p(score), _p(ff_idx), _p(y), act)
    return {"y": y, "in_idx": in_idx, "score": score, "ff_idx": ff_idx}


def add_rmsnorm(x, y, dtype: int, eps: float = 1e-6):
    """Residual add then unit-gain RMSNorm between stacked layers, fp64."""
    x = _u16(np.atleast_2d(x)); y = _u16(np.atleast_2d(y))
    B, d = x.shape
    out = np.empty((B, d))
    lib().oracle_add_rmsnorm(_p(x), _p(y), dtype, B, d, float(eps), _p(out))
    return out


def max_threads() -> int:
    return int(lib().oracle_max_threads())


# ---------------------------------------------------------------------------
# Threshold mode (Sec. 4.1 masks with layer-wise thresholds, App. A.6) and
# its calibration (App. A.7, Alg. 1)
# ---------------------------------------------------------------------------

def double_to_bf16(v: float) -> int:
    """bfloat16 round-to-nearest-even of a double (bit pattern)."""
    return int(lib().oracle_double_to_bf16(float(v)))


def halves_to_double(bits, dtype: int):
    """Exact values of an array of 16-bit patterns."""
    h = _u16(bits)
    out = np.empty(h.shape)
    lib().oracle_halves_to_double(_p(h), h.size, dtype, _p(out))
    return out


def round_to_dtype(v, dtype: int):
    """Array of doubles rounded (RNE) to the 16-bit dtype, as uint16 bits."""
    v = np.ascontiguousarray(v, dtype=np.float64)
    out = np.empty(v.shape, np.uint16)
    lib().oracle_round_to_dtype(_p(v), v.size, dtype, _p(out))
    return out


def select_threshold(key, tau: float):
    """App. A.6 threshold rule: ascending indices with key >= tau."""
    key = np.ascontiguousarray(key, dtype=np.float64)
    out = np.empty(max(key.size, 1), np.int32)
    k = lib().oracle_select_threshold(_p(key), key.size, float(tau), _p(out))
    return out[:k].copy()


def select_inputs_tau(x, dtype: int, tau_x: float):
    """Sec. 4.1 input mask with a threshold: max_b |x_{b,i}| >= tau_x."""
    x = _u16(np.atleast_2d(x))
    B, d = x.shape
    out = np.empty(d, np.int32)
    k = lib().oracle_select_inputs_tau(_p(x), dtype, B, d, float(tau_x), _p(out))
    return out[:k].copy()


def ffn_sparse_tau(x, dtype: int, w_gate, w_up, w_down, tau_x: float, tau_s: float, *,
                   codes_g=None, scales_g=None, codes_u=None, scales_u=None, group: int = 0,
                   kind=PROXY_QUANT, mask_override=None, act=SILU):
    """Whole Sec. 4.1 decode step with thresholds.  Returns dict(y, in_idx,
    score, ff_idx, k_in, k_ff); the counts follow from the data."""
    x = _u16(np.atleast_2d(x))
    B, d = x.shape
    wg, wu, wd = _u16(w_gate), _u16(w_up), _u16(w_down)
    f = wg.shape[0]
    if kind == PROXY_QUANT:
        codes_g = np.ascontiguousarray(codes_g, np.int8)
        codes_u = np.ascontiguousarray(codes_u, np.int8)
        scales_g, scales_u = _u16(scales_g), _u16(scales_u)
    mo = None if mask_override is None else np.ascontiguousarray(mask_override, np.int32)
    in_idx = np.empty(d, np.int32)
    score = np.empty(f)
    ff_idx = np.empty(f, np.int32)
    counts = np.zeros(2, np.int32)
    y = np.empty((B, d))
    lib().oracle_ffn_sparse_tau(_p(x), dtype, B, d, f, _p(wg), _p(wu), _p(wd), kind,
                                _p(codes_g), _p(scales_g), _p(codes_u), _p(scales_u), group,
                                float(tau_x), float(tau_s), _p(mo), 0 if mo is None else mo.size,
                                _p(in_idx), _p(score), _p(ff_idx), _p(counts), _p(y), act)
    k_in, k_ff = int(counts[0]), int(counts[1])
    return {"y": y, "in_idx": in_idx[:k_in].copy(), "score": score,
            "ff_idx": ff_idx[:k_ff].copy(), "k_in": k_in, "k_ff": k_ff}


class Reservoir:
    """App. A.7 bounded activation sample (Algorithm R); the caller supplies
    one uniform 64-bit random number per offered value."""

    def __init__(self, cap: int):
        self.cap = int(cap)
        self.buf = np.zeros(self.cap)
        self.seen = ctypes.c_longlong(0)

    def add(self, values, rand_u64):
        v = np.ascontiguousarray(values, dtype=np.float64).ravel()
        r = np.ascontiguousarray(rand_u64, dtype=np.uint64).ravel()
        assert r.size == v.size
        lib().oracle_reservoir_add(_p(self.buf), self.cap, ctypes.byref(self.seen), _p(v),
                                   v.size, _p(r))

    def sample(self):
        return self.buf[:min(self.cap, self.seen.value)].copy()


def quantile_threshold(samples, s: float) -> float:
    """App. A.7 threshold for target sparsity s: the ascending sample value at
    position min(n - 1, floor(s n))."""
    v = np.ascontiguousarray(samples, dtype=np.float64).ravel()
    return float(lib().oracle_quantile_threshold(_p(v), v.size, float(s)))


def stack_layer_tau(x_bits, dtype: int, layer: dict, tau_x: float, tau_s: float,
                    eps: float = 1e-6):
    """One layer of the stacked model with the threshold rule: y = FFN(x),
    then x' = RMSNorm(x + y), each rounded once to the dtype.  Returns
    (x' bits [B][d], ffn_sparse_tau result)."""
    r = ffn_sparse_tau(x_bits, dtype, layer["w_gate"], layer["w_up"], layer["w_down"],
                       tau_x, tau_s, codes_g=layer["codes_g"], scales_g=layer["scales_g"],
                       codes_u=layer["codes_u"], scales_u=layer["scales_u"],
                       group=layer["group"], act=layer.get("act", SILU))
    y_bits = round_to_dtype(r["y"], dtype)
    xn = add_rmsnorm(x_bits, y_bits, dtype, eps)
    return round_to_dtype(xn, dtype), r


def calibrate_stack(tokens, dtype: int, layers, s1: float, s2: float, cap: int, draw,
                    eps: float = 1e-6):
    """Alg. 1 sequential threshold calibration on calibration tokens.

    tokens: [T][d] bit patterns (the first layer's inputs, one token a row).
    layers: per layer dict(w_gate, w_up, w_down, codes_g, scales_g, codes_u,
    scales_u, group).  For each layer in depth order: collect its inputs
    through the earlier layers run with their finalised thresholds, set
    tau_x from |x| (target s1), build m_x per token, set tau_s from the proxy
    |s~| computed on m_x (target s2), then finalise the layer.  Samples go
    through a reservoir of `cap`; draw(n) returns n uniform uint64 draws.
    Returns [(tau_x, tau_s)] per layer."""
    xs = _u16(np.atleast_2d(tokens))
    T, d = xs.shape
    taus = []
    for layer in layers:
        res_x = Reservoir(cap)
        for t in range(T):
            mag = np.abs(halves_to_double(xs[t], dtype))
            res_x.add(mag, draw(mag.size))
        tau_x = quantile_threshold(res_x.sample(), s1)
        res_s = Reservoir(cap)
        for t in range(T):
            in_idx = select_inputs_tau(xs[t], dtype, tau_x)
            _, _, st, _ = proxy(xs[t], dtype, in_idx, codes_g=layer["codes_g"],
                                scales_g=layer["scales_g"], codes_u=layer["codes_u"],
                                scales_u=layer["scales_u"], group=layer["group"],
                                act=layer.get("act", SILU))
            mag = np.abs(st[0])
            res_s.add(mag, draw(mag.size))
        tau_s = quantile_threshold(res_s.sample(), s2)
        taus.append((tau_x, tau_s))
        xs = np.stack([stack_layer_tau(xs[t], dtype, layer, tau_x, tau_s, eps)[0][0]
                       for t in range(T)])
    return taus


# ---------------------------------------------------------------------------
# Cost model and sparsity allocation (Sec. 4.2)
# ---------------------------------------------------------------------------

def prox_cost(s1: float, s2: float, alpha: float = 1.0 / 3.0) -> float:
    """Sec. 4.2 normalised cost (a dense FFN costs 3)."""
    return float(lib().oracle_prox_cost(s1, s2, alpha))


def effective_sparsity(s1: float, s2: float, alpha: float = 1.0 / 3.0) -> float:
    """Sec. 4.2 effective sparsity against the dense FFN."""
    return float(lib().oracle_effective_sparsity(s1, s2, alpha))


def allocate(e: float, alpha: float = 1.0 / 3.0, s_ref: float = 0.7, s1_min: float = 0.0,
             s1_max: float = 0.7):
    """Sec. 4.2 allocation of a target effective sparsity: (s1, s2)."""
    a, b = ctypes.c_double(), ctypes.c_double()
    lib().oracle_allocate(e, alpha, s_ref, s1_min, s1_max, ctypes.byref(a), ctypes.byref(b))
    return a.value, b.value


def gate_act(z: float, act: int) -> float:
    """Gate activation: SiLU (SwiGLU, Sec. 2.1) or GELU z Phi(z) (GeGLU)."""
    return float(lib().oracle_gate_act(float(z), int(act)))
