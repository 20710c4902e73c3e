"""GPU parity over seeded random small parameter sets: ring size, prime counts,
digit width (so every transform split, short last digits, one to eight digits
and the ModUp / ModDown target grouping meet), block shape and row counts.
Each set checks two rotations and a diagonal block product word for word
against the oracle, and the decrypted scores against float64."""
import numpy as np
import pytest

from oracle import ckks
from paper_2608_21131_amd import gen

from common import PARAMS, Pair, say

pytestmark = pytest.mark.gpu


def _sets(count=10, seed=2608):
    g = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        logn = int(g.integers(10, 14))
        K = int(g.integers(1, 5))
        L = int(g.integers(2, 17))
        if -(-L // K) > 8:
            continue
        d = int(g.choice([16, 32, 64]))
        B = int(g.choice([b for b in (2, 4, 8) if d % b == 0]))
        nblk = int(g.integers(1, 3))
        rows = [int(g.integers(1, (1 << logn) // 2 + 1)) for _ in range(nblk)]
        steps = sorted({1, int(g.integers(2, (1 << logn) // 2))})
        out.append((logn, L, K, d, B, rows, steps))
    return out


SETS = _sets()


@pytest.mark.parametrize("cfg", SETS, ids=[f"n{c[0]}-L{c[1]}-K{c[2]}-d{c[3]}-B{c[4]}" for c in SETS])
def test_random_parameter_sets(cfg):
    logn, L, K, d, B, rows_list, steps = cfg
    name = f"sweep_{logn}_{L}_{K}"
    PARAMS[name] = (logn, L, K)
    p = Pair(name, wid=21)
    S = p.par.slots
    say(f"[sweep] N=2^{logn} L={L} K={K} dnum={p.par.dnum} d={d} B={B} rows={rows_list} steps={steps}")
    # rotations
    v = np.random.default_rng(logn * 100 + L).uniform(-1, 1, S)
    ct_dev, ct_orc = p.encrypt_both(ckks.encode(v, p.n, 40), tag=21)
    keys = p.keys(steps)
    for r in steps:
        got = p.export_ct(p.ctx.rotate(ct_dev, r))[0]
        assert np.array_equal(got, p.orc.rotate(ct_orc, r, keys[r])), r
    # a diagonal block product (baby steps, multiply-accumulate, giant steps)
    G = d // B
    g = gen.rng(21, gen.STREAM_DB, d, B)
    Xs = [gen.gaussian_unit_rows(g, r, d) for r in rows_list]
    q = gen.gaussian_unit_rows(gen.rng(21, gen.STREAM_QUERY), 1, d)[0]
    ct_dev, ct_orc = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=22)
    keys = p.keys(ckks.steps_for_bsgs(d, B))
    coeffs = [ckks.layout_b_coeffs(X, p.par, d, B) for X in Xs]
    blocks = [p.ctx.encode_db_block_int(c) for c in coeffs]
    out = p.ctx.score_block(ct_dev, blocks, d, 1, B)
    got = p.export_ct(out, len(Xs))
    qrot = p.orc.baby_rotations(ct_orc, B, keys)
    for i, (X, c) in enumerate(zip(Xs, coeffs)):
        pts = np.stack([ckks.to_residues(ci, p.par.q) for ci in c]).reshape(G, B, p.par.L, p.n)
        assert np.array_equal(got[i], p.orc.bsgs_block(qrot, pts, B, G, keys)), i
        z = p.ctx.decode(p.ctx.decrypt(out[i * p.ctx.ct_words:(i + 1) * p.ctx.ct_words]), 80)
        assert np.max(np.abs(z[:len(X)] - X @ q)) < 1e-4


@pytest.mark.parametrize("cfg", SETS[:3], ids=[f"n{c[0]}-L{c[1]}-K{c[2]}-d{c[3]}-B{c[4]}" for c in SETS[:3]])
def test_random_sets_query_batch(cfg):
    """Five queries prepared together and scored in one batch against four blocks: 20 blocks of
    giant steps (a 16-block chunk and a 4-block one), a four-query and a one-query plaintext pass.
    Every output equals the single-query path word for word (that path is checked against the
    oracle above)."""
    logn, L, K, d, B, _, _ = cfg
    name = f"sweep_{logn}_{L}_{K}"
    PARAMS[name] = (logn, L, K)
    p = Pair(name, wid=23)
    S = p.par.slots
    g = gen.rng(23, gen.STREAM_DB, d, B)
    blocks = [p.ctx.encode_db_block_int(ckks.layout_b_coeffs(gen.gaussian_unit_rows(g, r, d), p.par, d, B))
              for r in (S, S // 2, 7, S)]
    p.keys(ckks.steps_for_bsgs(d, B), oracle=False)
    qv = gen.gaussian_unit_rows(gen.rng(23, gen.STREAM_QUERY), 5, d)
    cts = [p.encrypt_both(ckks.encode(ckks.replicate(v, S), p.n, 40), tag=30 + j)[0] for j, v in enumerate(qv)]
    say(f"[sweep batch] N=2^{logn} L={L} K={K} d={d} B={B}: 5 queries x 4 blocks")
    preps = p.ctx.prepare_batch(cts, B)
    outs = p.ctx.score_batch(cts, preps, blocks, d, B)
    for j in range(5):
        single = p.ctx.score_block(cts[j], blocks, d, 1, B)
        assert np.array_equal(p.export_ct(outs[j], 4), p.export_ct(single, 4)), j
