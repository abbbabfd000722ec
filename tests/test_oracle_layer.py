"""Pins of the rest-of-layer oracle (the per-layer compute window around the
attention): exact cases where every product is a bfloat16 value, a
brute-force loop on tiny inputs, torch's own SiLU and bfloat16 rounding as
independent library routines, and invariants of the chain."""
import math

import numpy as np
import pytest
import torch

from oracle import layer


def _bits(x):
    return torch.tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _vals(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()


def test_rounding_matches_torch_nearest_even():
    # ties, near-ties, subnormals, huge values and signed zeros
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(4000) * 10.0 ** rng.integers(-30, 30, 4000),
                        [1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 2 ** -130, -0.0, 0.0, 3.0e38, 65504.0]])
    x32 = x.astype(np.float32).astype(np.float64)     # exactly representable in float32: one rounding only
    assert np.array_equal(layer.f64_to_bf16(x32), _bits(x32))
    assert layer.f64_to_bf16(np.array([1 + 2 ** -8]))[0] == 0x3F80      # tie to even: down
    assert layer.f64_to_bf16(np.array([1 + 3 * 2 ** -8]))[0] == 0x3F82  # tie to even: up


def _nearest_even_brute_force(x: float) -> int:
    """bfloat16 bits of float64 x by exhaustive search: the non-negative
    finite bfloat16 patterns 0x0000..0x7F7F increase with their value, so
    the two neighbours of |x| are found by bisection over all of them; their
    distances to |x| are compared in exact rational arithmetic, a tie goes
    to the even pattern.  0x7F80 (infinity) stands at 2^128 for rounding."""
    from fractions import Fraction
    if math.isnan(x):
        return 0x7FC0
    sign = 0x8000 if math.copysign(1.0, x) < 0 else 0
    a = abs(x)
    if a >= 2.0 ** 128:
        return sign | 0x7F80
    pats = np.arange(0x7F81, dtype=np.uint32)
    vals = (pats << 16).view(np.float32).astype(np.float64)
    vals[0x7F80] = 2.0 ** 128
    hi = int(np.searchsorted(vals, a, side="left"))      # first value >= |x|
    if vals[hi] == a:
        return sign | hi
    lo = hi - 1
    dlo, dhi = Fraction(a) - Fraction(float(vals[lo])), Fraction(float(vals[hi])) - Fraction(a)
    pick = lo if dlo < dhi else hi if dhi < dlo else (lo if lo % 2 == 0 else hi)
    return sign | pick


def test_rounding_is_one_step_from_float64():
    # values next to bfloat16 ties, where rounding first to float32 and then
    # to bfloat16 lands on the wrong side: 1 + 2^-8 + 2^-30 lies above the
    # tie between 0x3F80 and 0x3F81 by less than float32 can hold
    assert layer.f64_to_bf16(np.array([1 + 2 ** -8 + 2 ** -30]))[0] == 0x3F81
    assert layer.f64_to_bf16(np.array([1 + 2 ** -8 - 2 ** -30]))[0] == 0x3F80
    assert layer.f64_to_bf16(np.array([-(1 + 3 * 2 ** -8 - 2 ** -40)]))[0] == 0xBF81
    # subnormal ties: half the smallest subnormal goes to zero, 1.5 of it to 2 units
    assert layer.f64_to_bf16(np.array([2.0 ** -134, 3 * 2.0 ** -134, 2.0 ** -134 * (1 + 2 ** -30)])).tolist() == \
        [0x0000, 0x0002, 0x0001]
    # overflow: the largest finite value plus just under half its spacing stays finite
    big = float((np.uint32(0x7F7F) << 16).view(np.float32))
    assert layer.f64_to_bf16(np.array([big + 2.0 ** 119 * (1 - 2 ** -20), big + 2.0 ** 119, np.inf, -np.inf,
                                       np.nan])).tolist() == [0x7F7F, 0x7F80, 0x7F80, 0xFF80, 0x7FC0]
    # brute force over random values and values within 2^-20 .. 2^-50 relative of a tie
    rng = np.random.default_rng(5)
    xs = list(rng.standard_normal(300) * 2.0 ** rng.integers(-140, 130, 300))
    for b in rng.integers(0, 0x7F7F, 120):
        v = float((np.uint32(b) << 16).view(np.float32))
        nxt = float((np.uint32(b + 1) << 16).view(np.float32))
        tie = (v + nxt) / 2                       # exact in float64
        k = int(rng.integers(20, 51))
        xs += [tie, tie * (1 + 2.0 ** -k), tie * (1 - 2.0 ** -k), -tie * (1 + 2.0 ** -k)]
    xs += [0.0, -0.0, 2.0 ** -133, 2.0 ** -126 * (1 - 2 ** -9)]
    got = layer.f64_to_bf16(np.array(xs, dtype=np.float64)).tolist()
    want = [_nearest_even_brute_force(float(x)) for x in xs]
    assert got == want


def test_silu_special_values_and_torch():
    assert layer.silu(np.array([0.0]))[0] == 0.0
    assert abs(layer.silu(np.array([50.0]))[0] - 50.0) < 1e-12
    assert abs(layer.silu(np.array([-50.0]))[0]) < 1e-19
    assert layer.silu(np.array([math.log(3.0)]))[0] == pytest.approx(math.log(3.0) * 0.75, rel=1e-15)  # 1/(1+1/3)
    x = np.linspace(-12, 12, 1001)
    assert np.allclose(layer.silu(x), torch.nn.functional.silu(torch.tensor(x)).numpy(), rtol=1e-14, atol=1e-300)


def _chain_inputs(rng, T, H, F, NQ, int_valued=False):
    def mat(shape, scale):
        if int_valued:
            return _bits(rng.integers(-3, 4, shape).astype(np.float32))
        return _bits((rng.standard_normal(shape) * scale).astype(np.float32))
    return (mat((T, H), 1.0), mat((H, H), H ** -0.5), mat((H, 2 * F), H ** -0.5), mat((F, H), F ** -0.5),
            mat((H, NQ), H ** -0.5))


def test_identity_and_permutation_weights_pass_values_through():
    rng = np.random.default_rng(1)
    T, H = 5, 8
    A = _bits(rng.standard_normal((T, H)).astype(np.float32))
    perm = rng.permutation(H)
    P = np.zeros((H, H), np.float32)
    P[np.arange(H), perm] = 1.0                      # column perm[i] takes input feature i
    eye = _bits(np.eye(H, dtype=np.float32))
    wgu = _bits(np.concatenate([np.eye(H), np.eye(H)], axis=1).astype(np.float32))
    out = layer.rest_of_layer(A, _bits(P), wgu, eye, eye)
    assert np.array_equal(out["o"][:, perm], A)
    assert np.array_equal(out["gu"][:, :H], out["o"]) and np.array_equal(out["gu"][:, H:], out["o"])
    g = _vals(out["o"])
    want = torch.nn.functional.silu(torch.tensor(g)) * torch.tensor(g)
    assert np.array_equal(out["act"], want.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16))
    assert np.array_equal(out["h"], out["act"]) and np.array_equal(out["qkv"], out["act"])


def test_brute_force_loops_on_tiny_integer_inputs():
    # small integers: every GEMM sum is exact in float64 and in bfloat16
    # (|sum| <= 3*3*8*... stays below 256), so only the SiLU stage rounds
    rng = np.random.default_rng(2)
    T, H, F, NQ = 3, 4, 3, 6
    A, wo, wgu, wd, wq = _chain_inputs(rng, T, H, F, NQ, int_valued=True)
    a, Wo, Wgu, Wd, Wq = (_vals(m).tolist() for m in (A, wo, wgu, wd, wq))

    def mm(x, w):
        return [[sum(x[i][k] * w[k][j] for k in range(len(w))) for j in range(len(w[0]))] for i in range(len(x))]

    def rnd(m):
        bits = np.array([[_nearest_even_brute_force(v) for v in r] for r in m], dtype=np.uint16)
        return _vals(bits).tolist()

    o = mm(a, Wo)
    assert all(abs(v) < 256 for r in o for v in r)
    gu = mm(o, Wgu)
    act = rnd([[gu[i][j] / (1 + math.exp(-gu[i][j])) * gu[i][F + j] for j in range(F)] for i in range(T)])
    h = rnd(mm(act, Wd))
    qkv = rnd(mm(h, Wq))
    out = layer.rest_of_layer(A, wo, wgu, wd, wq)
    assert _vals(out["o"]).tolist() == o
    assert _vals(out["gu"]).tolist() == gu
    assert _vals(out["act"]).tolist() == act
    assert _vals(out["h"]).tolist() == h
    assert _vals(out["qkv"]).tolist() == qkv


def test_power_of_two_scaling_commutes_with_the_chain():
    # scaling W_down by 2 doubles h and qkv exactly (rounding commutes with x2)
    rng = np.random.default_rng(3)
    A, wo, wgu, wd, wq = _chain_inputs(rng, 7, 16, 24, 20)
    base = layer.rest_of_layer(A, wo, wgu, wd, wq)
    wd2 = _bits(_vals(wd) * 2.0)
    twice = layer.rest_of_layer(A, wo, wgu, wd2, wq)
    assert np.array_equal(twice["act"], base["act"])
    assert np.array_equal(_vals(twice["h"]), 2.0 * _vals(base["h"]))
    assert np.array_equal(_vals(twice["qkv"]), 2.0 * _vals(base["qkv"]))


def test_rows_are_independent():
    # each token's row goes through the chain on its own
    rng = np.random.default_rng(4)
    A, wo, wgu, wd, wq = _chain_inputs(rng, 9, 16, 24, 20)
    full = layer.rest_of_layer(A, wo, wgu, wd, wq)
    part = layer.rest_of_layer(A[[2, 7]], wo, wgu, wd, wq)
    for k in full:
        assert np.array_equal(part[k], full[k][[2, 7]])


def test_flop_count():
    # Llama 3.1 8B layer: H 4096, F 14336, QKV 6144 -> 218,103,808 weights
    assert layer.gemm_flops(1, 4096, 14336, 6144) == 2 * 218_103_808
