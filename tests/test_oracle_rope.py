"""Pins of the oracle's rotary position embeddings in the readout (pseudo-
tokens of prototype k share the rotary position tau_k; near tokens keep
their own positions).

Each test checks the rotation against something other than its own code:
complex multiplication, a block-diagonal rotation matrix, the relative-
position property that defines RoPE, and, end to end, exact attention over
the whole history with every key rotated at its own position (the capacity
limit, where each prototype is one token and tau_k is that token's
position).  No GPU is needed.
"""
import math

import numpy as np
import pytest

from oracle import protokv_oracle as O
from paper_2606_26762_amd import workloads as W
from tests.test_oracle_pins import _sdpa, tiny_params, tiny_stream

F32 = np.float32


def _complex_rope(x, pos, theta):
    """Rotate-half RoPE as complex multiplication: z_i = x_i + 1j x_(i+D/2)
    times exp(1j pos theta^(-2i/D))."""
    x = np.asarray(x, dtype=np.float64)
    h = x.shape[-1] // 2
    z = x[..., :h] + 1j * x[..., h:]
    w = np.exp(1j * np.asarray(pos, dtype=np.float64)[..., None] * theta ** (-np.arange(h) * 2.0 / (2 * h)))
    r = z * w
    return np.concatenate([r.real, r.imag], axis=-1)


def test_rotation_is_complex_multiplication_and_a_block_rotation_matrix():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 128))
    pos = np.array([0, 1, 7, 1000, 123457])
    got = O.rope_rotate(x, pos, 10000.0)
    assert np.allclose(got, _complex_rope(x, pos, 10000.0), atol=1e-12)
    # one vector through an explicit D x D rotation matrix
    D, h = 128, 64
    R = np.zeros((D, D))
    for i in range(h):
        a = 1000 * 10000.0 ** (-2.0 * i / D)
        R[i, i], R[i, i + h], R[i + h, i], R[i + h, i + h] = math.cos(a), -math.sin(a), math.sin(a), math.cos(a)
    assert np.allclose(O.rope_rotate(x[3], 1000, 10000.0), R @ x[3], atol=1e-12)


def test_position_zero_is_the_identity_and_norms_are_kept():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((4, 128))
    assert np.array_equal(O.rope_rotate(x, 0, 1e6), x)
    y = O.rope_rotate(x, np.array([3, 99, 4096, 10 ** 6]), 1e6)
    h = 64
    assert np.allclose(x[:, :h] ** 2 + x[:, h:] ** 2, y[:, :h] ** 2 + y[:, h:] ** 2, atol=1e-12)


@pytest.mark.parametrize("theta", [10000.0, 1e6])
def test_logits_depend_on_relative_position_only(theta):
    """<R(p) q, R(s) k> = <R(p + d) q, R(s + d) k> = <q, R(s - p) k>."""
    rng = np.random.default_rng(2)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    for p, s, d in ((5, 2, 1000), (0, 300, 77), (12345, 67, 999999)):
        a = O.rope_rotate(q, p, theta) @ O.rope_rotate(k, s, theta)
        b = O.rope_rotate(q, p + d, theta) @ O.rope_rotate(k, s + d, theta)
        c = q @ O.rope_rotate(k, s - p, theta)
        assert abs(a - b) <= 1e-9 * (1 + abs(a)) and abs(a - c) <= 1e-9 * (1 + abs(a))


@pytest.mark.parametrize("S", [1, 8])
def test_capacity_limit_with_rope_is_exact_positional_attention(S):
    """K >= evicted tokens: each prototype is one token, tau_k is its stream
    position f * T + j, so the readout is exact attention over the whole
    history with every key rotated (complex form) at its own position and
    query token t at P + t (P = frames * T); far logits shift by ln S."""
    p = tiny_params(capacity=64, S=S, rope_theta=10000.0)
    frames = 6
    wl = tiny_stream(p, frames, seed=9)
    cb = W.make_codebooks(wl, units=[0], samples=128, iters=2)
    gen = W.HostStream(wl, units=[0])
    st = O.OracleStream(p, [0], cb)
    ks, vs = [], []
    for _ in range(frames):
        k, v = gen.next_frame()
        ks.append(k[0])
        vs.append(v[0])
        st.append_frame(k, v)
    pseudo = st.synthesize()
    Tq = 8
    q = np.random.default_rng(0).standard_normal((1, Tq, 1, 128)).astype(F32)
    out, _ = st.attend(q, 1, pseudo)
    T = p.tokens_per_frame
    kall = np.concatenate(ks)
    kr = _complex_rope(kall, np.arange(len(kall)), 10000.0)
    qr = _complex_rope(q[0, :, 0, :], frames * T + np.arange(Tq), 10000.0)
    mask = np.zeros(len(kall))
    mask[: len(kall) - p.window_frames * T] = math.log(S)
    ref = _sdpa(qr, kr, np.concatenate(vs), mask)
    assert np.allclose(out[0, :, 0, :], ref, atol=1e-10)


def test_rotation_changes_the_readout():
    """The same stream read with and without RoPE gives different outputs
    (the rotation is applied, not skipped)."""
    p0 = tiny_params(capacity=16)
    pr = tiny_params(capacity=16, rope_theta=10000.0)
    frames = 5
    outs = []
    for p in (p0, pr):
        wl = tiny_stream(p, frames, seed=4)
        cb = W.make_codebooks(wl, units=[0], samples=128, iters=2)
        gen = W.HostStream(wl, units=[0])
        st = O.OracleStream(p, [0], cb)
        for _ in range(frames):
            st.append_frame(*gen.next_frame())
        q = np.random.default_rng(1).standard_normal((1, 4, 1, 128)).astype(F32)
        outs.append(st.attend(q, 1, st.synthesize())[0])
    assert not np.allclose(outs[0], outs[1])   # the rotation changes the readout
