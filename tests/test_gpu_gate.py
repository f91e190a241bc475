"""Test-time routing (Sec. 3.2.2) and the gated residual of Eq. 1 with its
gradient, through the C ABI, against the oracle.

Greedy routing: assign, perm and offsets bit-exact (argmax with the lowest
expert on ties; stable counting sort). Combine and backward: fp32 arithmetic
on the device against fp64 in the oracle; the bounds are a few fp32 rounding
steps of the magnitude sums involved, plus one bf16 rounding of each stored
bf16 output (rel 2^-8)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2103_16716_amd as pb
import workloads as wl
from gpu_common import dev, host, inputs_on_device

pytestmark = pytest.mark.gpu

F32_EPS = float(np.finfo(np.float32).eps)
BF16_REL = 2.0 ** -8


def as_f64(x: np.ndarray) -> np.ndarray:
    return wl.bf16_bits_to_f32(x).astype(np.float64) if x.dtype == np.uint16 else x.astype(np.float64)


def rand_rows(rng, T, d, dtype):
    x = rng.standard_normal((T, d), dtype=np.float32)
    return wl.f32_to_bf16_bits(x) if dtype == "bf16" else x


@pytest.mark.parametrize("name", ["t8192-e64-d1024", "t32768-e128-d2048-mix8"])
def test_greedy_routing_bit_exact(name):
    inp = wl.make_inputs(name)
    S = pb.affinity(*inputs_on_device(inp))
    a, perm, off = pb.greedy_assign(S)
    torch.cuda.synchronize()
    Sh = host(S)
    a_ref = oracle.greedy_argmax(Sh)
    np.testing.assert_array_equal(host(a), a_ref)
    np.testing.assert_array_equal(host(perm), oracle.stable_perm(a_ref, Sh.shape[1]))
    np.testing.assert_array_equal(host(off), oracle.expert_offsets(a_ref, Sh.shape[1]))


@pytest.mark.parametrize("T,E", [(1000, 70), (257, 3), (64, 1), (1, 5), (5000, 2048),
                                 (300000, 16), (4099, 512), (2000, 500), (3001, 513), (77, 130),
                                 (800000, 8)])
def test_greedy_routing_ragged(T, E):
    """Single-launch routing (E <= 512: several token passes per block at T =
    300000, the widest E, E/4 not a power of two, scalar loads for E % 4 != 0)
    and the multi-launch paths: count + place (E <= 512 with more tokens than
    192 blocks of 4096 hold, T = 800000) and count + scan + offsets + scatter
    (E > 512)."""
    rng = np.random.Generator(np.random.PCG64(T + E))
    S = rng.standard_normal((T, E), dtype=np.float32)
    S[::7, :] = np.round(S[::7, :])          # ties: the lowest expert must win
    S[T // 2, :] = -np.inf                   # a row with no finite score: expert 0
    S[T // 3, :] = -np.inf
    S[T // 3, E - 1] = 0.0
    a, perm, off = pb.greedy_assign(dev(S))
    a_ref = oracle.greedy_argmax(S)
    np.testing.assert_array_equal(host(a), a_ref)
    np.testing.assert_array_equal(host(perm), oracle.stable_perm(a_ref, E))
    np.testing.assert_array_equal(host(off), oracle.expert_offsets(a_ref, E))


def test_greedy_routing_reuses_a_workspace():
    """The workspace holds anything at the first call (here all bytes 0xA5)
    and one workspace serves calls of different shapes in a row; the results
    go to the caller's output tensors."""
    n = int(pb.lib().base_greedy_workspace_size(40000, 128))
    ws = torch.full((n,), 0xA5, dtype=torch.uint8, device="cuda")
    for T, E in ((40000, 128), (40000, 128), (1000, 64), (33333, 100)):
        rng = np.random.Generator(np.random.PCG64(7 * T + E))
        S = rng.standard_normal((T, E), dtype=np.float32)
        outs = [torch.full((n,), -7, dtype=torch.int32, device="cuda") for n in (T, T, E + 1)]
        a, perm, off = pb.greedy_assign(dev(S), workspace=ws, out_assign=outs[0],
                                        out_perm=outs[1], out_offsets=outs[2])
        assert all(x is y for x, y in zip((a, perm, off), outs))
        a_ref = oracle.greedy_argmax(S)
        np.testing.assert_array_equal(host(a), a_ref)
        np.testing.assert_array_equal(host(perm), oracle.stable_perm(a_ref, E))
        np.testing.assert_array_equal(host(off), oracle.expert_offsets(a_ref, E))


def _routing(kind, S):
    if kind == "balanced":
        r = pb.assign(S)
        T, E = S.shape
        return r.assign, r.perm, pb.balanced_offsets(T, E, S.device)
    return pb.greedy_assign(S)


@pytest.mark.parametrize("dtype,name,kind", [("bf16", "t4096-e16-d512", "balanced"),
                                             ("bf16", "t4096-e16-d512", "greedy"),
                                             ("f32", "t512-e8-d128-f32", "balanced"),
                                             ("f32", "t512-e8-d128-f32", "greedy")])
def test_gate_combine_against_oracle(dtype, name, kind):
    inp = wl.make_inputs(name)
    T, d = inp.wl.T, inp.wl.d
    Hd, Wd = inputs_on_device(inp)
    S = pb.affinity(Hd, Wd)
    a, perm, _ = _routing(kind, S)
    rng = np.random.Generator(np.random.PCG64(7))
    F = rand_rows(rng, T, d, dtype)
    Y = pb.gate_combine(dev(F), Hd, S, a, perm)
    torch.cuda.synchronize()
    ref = oracle.gate_combine(as_f64(F), as_f64(inp.H_store), host(S).astype(np.float64),
                              host(a), host(perm))
    mag = np.abs(oracle.gate_combine(np.abs(as_f64(F)), np.abs(as_f64(inp.H_store)),
                                     host(S).astype(np.float64), host(a), host(perm)))
    err = np.abs(as_f64(host(Y)) - ref)
    bound = 8 * F32_EPS * mag + (BF16_REL * np.abs(ref) if dtype == "bf16" else 0.0) + 1e-30
    assert np.all(err <= bound), float((err / bound).max())


@pytest.mark.parametrize("dtype,name,kind", [("bf16", "t4096-e16-d512", "balanced"),
                                             ("bf16", "t4096-e16-d512", "greedy"),
                                             ("f32", "t512-e8-d128-f32", "balanced"),
                                             ("f32", "t512-e8-d128-f32", "greedy")])
def test_gate_backward_against_oracle(dtype, name, kind):
    inp = wl.make_inputs(name)
    T, E, d = inp.wl.T, inp.wl.E, inp.wl.d
    Hd, Wd = inputs_on_device(inp)
    S = pb.affinity(Hd, Wd)
    a, perm, off = _routing(kind, S)
    rng = np.random.Generator(np.random.PCG64(11))
    F = rand_rows(rng, T, d, dtype)
    dY = rand_rows(rng, T, d, dtype)
    dH, dF, dW, dS = pb.gate_backward(dev(dY), dev(F), Hd, Wd, S, a, perm, off)
    torch.cuda.synchronize()
    Sh = host(S).astype(np.float64)
    ah, ph = host(a), host(perm)
    Fh, dYh, Hh, Wh = as_f64(F), as_f64(dY), as_f64(inp.H_store), as_f64(inp.W_store)
    rH, rF, rW, rS = oracle.gate_backward(dYh, Fh, Hh, Wh, Sh, ah, ph)
    g = oracle.gate.sigmoid(Sh[np.arange(T), ah])
    f_tok = oracle.scatter(Fh, ph)
    # dS: an fp32 dot product of length d, then the gate derivative
    dot_mag = g * (1 - g) * np.sum(np.abs(dYh * f_tok), axis=1)
    assert np.all(np.abs(host(dS) - rS) <= 4 * d * F32_EPS * dot_mag + 8 * F32_EPS * np.abs(rS) + 1e-30)
    bf = BF16_REL if dtype == "bf16" else 0.0
    # dF = g dY (routed order)
    eF = np.abs(as_f64(host(dF)) - rF)
    assert np.all(eF <= 8 * F32_EPS * np.abs(rF) + bf * np.abs(rF) + 1e-30)
    # dH = dY + dS W[a]: dS's error times |W| plus roundings
    dS_err = 4 * d * F32_EPS * dot_mag + 8 * F32_EPS * np.abs(rS)
    magH = np.abs(dYh) + np.abs(rS)[:, None] * np.abs(Wh[ah])
    eH = np.abs(as_f64(host(dH)) - rH)
    assert np.all(eH <= 8 * F32_EPS * magH + dS_err[:, None] * np.abs(Wh[ah]) + bf * np.abs(rH) + 1e-30)
    # dW[e] = sum over the expert's tokens of dS_t h_t, accumulated in fp32:
    # the sum's rounding (count steps) plus the propagated error of each dS_t
    counts = np.bincount(ah, minlength=E)
    magW = np.zeros((E, d))
    np.add.at(magW, ah, np.abs(rS)[:, None] * np.abs(Hh))
    propW = np.zeros((E, d))
    np.add.at(propW, ah, dS_err[:, None] * np.abs(Hh))
    eW = np.abs(host(dW).astype(np.float64) - rW)
    assert np.all(eW <= (counts[:, None] + 8) * F32_EPS * magW + propW + 1e-30)
