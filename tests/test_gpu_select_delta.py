"""np_select_delta -- np_select followed by np_delta in one call (Sec. 3.4:
the fixed-size active set of every layer and its delta against the resident
set) -- against the two separate calls and against the oracle's O2 and O3.

Bar: bit for bit.  The mask, the active ids, the three state arrays, every
defined entry of the delta lists and the error word must equal those of the
two calls on the same inputs, and the ids and the delta must equal the
oracle's, run on the same fp32 scores.  Shapes cover the fused kernel (F up
to 16384, C up to 8192, k up to 4096: the 7B and 13B layer shapes, the edge
of each limit, F not a multiple of 4 or of 32, C not a multiple of 32) and
the shapes that fall back to the two kernels (F above the limit, k above it).
Scores follow an AR(1) sequence across tokens, so consecutive active sets
overlap and the resident buffer fills, evicts and reuses slots; some tokens
quantise the scores to a few levels so that the k-th score is tied many
times over, and some carry -0.0 and +0.0.
"""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import binding as B
from paper_2608_22643_amd import workload as W
from gpu_util import Bufs, compare_delta, from_dev, say

pytestmark = pytest.mark.gpu


def cfg_small(name, L, d, F, k, C):
    return W.Config(name, L, d, F, 8, k / F, C / F, "f32", "f32", 4, rho_given=0.9, k_override=k,
                    c_override=C)


SHAPES = {
    "tiny": W.get("tiny"),
    "ragged": cfg_small("ragged", 3, 64, 1000, 100, 300),      # F % 32 != 0, F % 4 == 0
    "odd_f": cfg_small("odd_f", 2, 64, 11001, 1650, 5000),     # F % 4 != 0: scalar score loads
    "k_one": cfg_small("k_one", 2, 64, 333, 1, 5),
    "k_eq_c": cfg_small("k_eq_c", 2, 64, 640, 64, 64),
    "k_eq_f": cfg_small("k_eq_f", 2, 64, 96, 96, 96),
    "7b_layers": cfg_small("7b_layers", 4, 64, 11008, 1651, 5504),
    "13b_layers": cfg_small("13b_layers", 3, 64, 13824, 1658, 5529),  # C % 32 != 0
    "fused_max": cfg_small("fused_max", 2, 64, 16384, 4096, 8192),
    "f_over": cfg_small("f_over", 2, 64, 16385, 2000, 6000),   # two kernels
    "k_over": cfg_small("k_over", 2, 64, 14336, 4097, 8192),   # two kernels
}


def score_sequence(rng, L, F, T):
    """[T][L][F] fp32: AR(1) over tokens (rho 0.95); every third token
    quantised to 8 levels (long ties at the k-th score); signed zeros."""
    s = rng.standard_normal((L, F))
    out = []
    for t in range(T):
        s = 0.95 * s + np.sqrt(1 - 0.95 ** 2) * rng.standard_normal((L, F))
        v = s.astype(np.float32)
        if t % 3 == 2:
            v = (np.round(v * 2.0) / 2.0).astype(np.float32)
        v[:, ::97] = np.float32(0.0)
        v[:, 5::97] = np.float32(-0.0)
        out.append(v)
    return out


def run_pair(cfg, scores_seq, token_auto=False, corrupt_at=None):
    """Both paths over the sequence; after each token compares them with
    each other and (unless the state was corrupted) with the oracle."""
    L, F, C, k = cfg.layers, cfg.d_ffn, cfg.capacity, cfg.k
    a, b = Bufs(cfg), Bufs(cfg)
    a.reset()
    b.reset()
    st = orc.State(L, F, C)
    for t, sc in enumerate(scores_seq):
        if corrupt_at is not None and t == corrupt_at:
            # slot 0 (in use since the first token) names a neuron that does
            # not map back to it
            for bufs in (a, b):
                Q = bufs.neuron_of.view(L, C)
                Q[0, 0] = (int(Q[0, 0]) + 1) % F
        dev = torch.from_numpy(sc.reshape(-1)).cuda()
        a.scores.copy_(dev)
        b.scores.copy_(dev)
        B.np_select(a.shape, a.scores, a.mask, a.ids, a.ws)
        B.np_delta(a.shape, t, a.ids, a.state, a.out, a.ws)
        B.np_select_delta(b.shape, B.NP_TOKEN_AUTO if token_auto else t, b.scores, b.mask, b.ids,
                          b.state, b.out, b.ws)
        torch.cuda.synchronize()
        assert torch.equal(a.mask, b.mask), t
        assert torch.equal(a.ids, b.ids), t
        for x, y in zip(a.host_state(), b.host_state()):
            assert np.array_equal(x, y), t
        la, lb = a.host_lists(), b.host_lists()
        compare_delta(lb, la, L)
        ea, eb = B.np_device_error(a.ws), B.np_device_error(b.ws)
        assert ea == eb, (t, ea, eb)
        if corrupt_at is None:
            assert eb == 0
            _, ids = orc.select(sc, k)
            assert np.array_equal(from_dev(b.ids, np.int32, (L, k)), ids), t
            ref = orc.delta(t, ids, st, C)
            compare_delta(lb, ref, L)
    return a, b


@pytest.mark.parametrize("name", list(SHAPES))
def test_select_delta_matches_two_calls_and_oracle(name):
    cfg = SHAPES[name]
    say(f"[select_delta] {name} L'={cfg.layers} F={cfg.d_ffn} k={cfg.k} C={cfg.capacity}")
    rng = np.random.default_rng(cfg.d_ffn + cfg.k)
    run_pair(cfg, score_sequence(rng, cfg.layers, cfg.d_ffn, 8))


@pytest.mark.parametrize("name", ["7b_layers", "f_over"])
def test_select_delta_token_counter(name):
    """NP_TOKEN_AUTO: the step counter in the workspace gives tokens 0, 1, ...
    and is advanced after each call, as np_delta's."""
    cfg = SHAPES[name]
    say(f"[select_delta] token counter {name}")
    rng = np.random.default_rng(3)
    run_pair(cfg, score_sequence(rng, cfg.layers, cfg.d_ffn, 5), token_auto=True)


@pytest.mark.parametrize("name", ["7b_layers", "ragged"])
def test_select_delta_nan_and_corrupt_state(name):
    """A NaN score (NP_DEVERR_NAN_SCORE) and a corrupted slot map
    (NP_DEVERR_STATE) are reported exactly as by the two calls, and every
    output still equals theirs."""
    cfg = SHAPES[name]
    say(f"[select_delta] error cases {name}")
    rng = np.random.default_rng(4)
    seq = score_sequence(rng, cfg.layers, cfg.d_ffn, 4)
    seq[1][0, 11] = np.float32("nan")
    a, b = run_pair(cfg, seq, corrupt_at=3)
    assert B.np_device_error(b.ws) & B.NP_DEVERR_NAN_SCORE
    assert B.np_device_error(b.ws) & B.NP_DEVERR_STATE


def test_select_delta_hint_misses_and_stale_hints():
    """The fused kernel starts each layer's selection from the previous
    token's k-th key (a window kept in the workspace) and falls back to the
    full radix select when the k-th key lies outside it.  Scores that jump in
    scale and offset from token to token force the fallback; hints
    overwritten with arbitrary values (the workspace's control block holds
    them from byte 512, two words per layer) must not change any result."""
    cfg = SHAPES["7b_layers"]
    say("[select_delta] hint misses and stale hints")
    rng = np.random.default_rng(9)
    seq = score_sequence(rng, cfg.layers, cfg.d_ffn, 8)
    for t in range(1, 8, 2):  # every other token far from the previous one
        seq[t] = (seq[t] * np.float32(37.0) + np.float32(5.0)).astype(np.float32)
    run_pair(cfg, seq)

    L, F, C, k = cfg.layers, cfg.d_ffn, cfg.capacity, cfg.k
    a, b = Bufs(cfg), Bufs(cfg)
    a.reset()
    b.reset()
    st = orc.State(L, F, C)
    for t, sc in enumerate(score_sequence(np.random.default_rng(10), L, F, 6)):
        junk = rng.integers(0, 2**32, size=2 * L, dtype=np.uint64).astype(np.uint32)
        if t == 3:
            junk[1::2] = 0  # zero half-widths: no window
        b.ws[512: 512 + 8 * L].copy_(torch.from_numpy(junk.view(np.uint8)).cuda())
        dev = torch.from_numpy(sc.reshape(-1)).cuda()
        a.scores.copy_(dev)
        b.scores.copy_(dev)
        B.np_select(a.shape, a.scores, a.mask, a.ids, a.ws)
        B.np_delta(a.shape, t, a.ids, a.state, a.out, a.ws)
        B.np_select_delta(b.shape, t, b.scores, b.mask, b.ids, b.state, b.out, b.ws)
        torch.cuda.synchronize()
        assert torch.equal(a.mask, b.mask) and torch.equal(a.ids, b.ids), t
        _, ids = orc.select(sc, k)
        assert np.array_equal(from_dev(b.ids, np.int32, (L, k)), ids), t
        compare_delta(b.host_lists(), orc.delta(t, ids, st, C), L)
    assert B.np_device_error(b.ws) == 0
