"""Pins of the per-sequence-plan batch in the oracle (plan.batched_arena_bases,
cache.compress_arena_batched, cache.decode_step_batched, plan.read_bytes_batched)."""
import numpy as np

from oracle import cache as OC
from oracle import plan as P

A = P.Action


def _dims(B=3, L=4):
    return P.Dims(P.GQA, L, 4, 2, 64, batch=B, max_tokens=80)


def _inputs(dims, n, seed):
    rng = np.random.default_rng(seed)
    Ks = [rng.standard_normal((dims.batch, dims.n_kv_heads, n, dims.head_dim)).astype(np.float32)
          for _ in range(dims.n_layers)]
    Vs = [rng.standard_normal((dims.batch, dims.n_kv_heads, n, dims.head_dim)).astype(np.float32)
          for _ in range(dims.n_layers)]
    q = rng.standard_normal((dims.n_layers, dims.batch, dims.n_q_heads, dims.head_dim))
    return Ks, Vs, q


def test_equal_plans_reduce_to_the_uniform_batch():
    dims = _dims()
    plan = [A(False, 4), A(True, 16), A(False, 8), A(True, 16)]
    Ks, Vs, q = _inputs(dims, 70, 1)
    ab = OC.compress_arena_batched(dims, [plan] * 3, Ks, Vs)
    au = OC.compress_arena(dims, plan, Ks, Vs)
    ob = OC.decode_step_batched(dims, [plan] * 3, ab, q, 70, 0.125)
    ou = OC.decode_step(dims, plan, au, q, 70, 0.125)
    assert np.array_equal(ob, ou)
    assert P.read_bytes_batched(dims, [plan] * 3, 0, 4, 70) == P.read_bytes(dims, plan, 0, 4, 70)


def test_sequences_are_independent():
    dims = _dims()
    plans = [[A(False, 4), A(True, 16), A(False, 8), A(True, 16)],
             [A(False, 16), A(False, 2), A(True, 16), A(True, 16)],
             [A(False, 8), A(False, 8), A(False, 4), A(False, 2)]]
    Ks, Vs, q = _inputs(dims, 70, 2)
    out = OC.decode_step_batched(dims, plans, OC.compress_arena_batched(dims, plans, Ks, Vs), q, 70, 0.125)
    plans2 = [plans[0], [A(False, 2), A(True, 16), A(True, 16), A(False, 16)], plans[2]]
    Ks2 = [K.copy() for K in Ks]
    Ks2[0][1] += 1.0
    out2 = OC.decode_step_batched(dims, plans2, OC.compress_arena_batched(dims, plans2, Ks2, Vs), q, 70, 0.125)
    assert np.array_equal(out[:, [0, 2]], out2[:, [0, 2]])
    assert not np.array_equal(out[:, 1], out2[:, 1])
    # each sequence alone, as a one-sequence batch with its own plan
    sd = P.sequence_dims(dims)
    for b in range(3):
        a1 = OC.compress_arena(sd, plans[b], [K[b:b + 1] for K in Ks], [V[b:b + 1] for V in Vs])
        assert np.array_equal(out[:, b:b + 1], OC.decode_step(sd, plans[b], a1, q[:, b:b + 1], 70, 0.125))


def test_bases_are_aligned_and_disjoint():
    dims = _dims(B=4)
    plans = [[A(False, b), A(True, 16), A(False, 2), A(False, 16)] for b in (2, 4, 8, 16)]
    bases, total = P.batched_arena_bases(dims, plans)
    sd = P.sequence_dims(dims)
    sizes = [P.arena_offsets(sd, pl)[1] for pl in plans]
    assert all(b % 256 == 0 for b in bases)
    assert all(bases[i] + sizes[i] <= bases[i + 1] for i in range(3))
    assert total == bases[-1] + P.round256(sizes[-1])
    assert P.read_bytes_batched(dims, plans, 0, 4, 70) == sum(P.read_bytes(sd, pl, 0, 4, 70) for pl in plans)
