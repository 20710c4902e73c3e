"""Parity at the workloads' full sizes, in the launch configuration bench.py
times: every GPU output ciphertext the oracle can afford is compared word for
word (the last, partial block of the multi-block levels), and every decrypted
score against float64 inner products (<= 1e-4)."""
import numpy as np
import pytest

from oracle import ckks
from paper_2608_21131_amd import workloads as wl

from common import say

pytestmark = pytest.mark.gpu


class Setup:
    """Library context + oracle with the workload's secret and keys."""

    def __init__(self, w: wl.Workload, oracle_steps=None):
        from paper_2608_21131_amd import fa
        self.w = w
        self.par = ckks.Params(logn=w.log_n, L=w.L, K=w.K)
        self.orc = ckks.Oracle(self.par)
        self.ctx = fa.Context(w.log_n, w.L, w.K, 40)
        assert self.ctx.primes == self.par.primes
        self.s = wl.secret(w)
        steps = wl.rotation_steps(w)
        say(f"[setup] {w.name}: {len(steps)} rotation keys")
        for i in range(0, len(steps), 8):
            chunk = steps[i:i + 8]
            rand = [wl.key_randomness(w, r, self.par.primes, self.par.dnum) for r in chunk]
            self.ctx.keygen(self.s, chunk, np.stack([x[0] for x in rand]), np.stack([x[1] for x in rand]))
        self.keys = {}
        for r in (steps if oracle_steps is None else oracle_steps):
            a, e = wl.key_randomness(w, r, self.par.primes, self.par.dnum)
            self.keys[r] = self.orc.keygen(self.s, r, a, e)

    def encrypt_query(self, v):
        a, e = wl.enc_randomness(self.w, self.par.q)
        m = ckks.encode(ckks.replicate(v, self.par.slots), self.par.n, 40)
        return self.ctx.encrypt(m, a, e), self.orc.encrypt(m, a, e, self.s)

    def decode(self, ct_tensor, i, log_scale):
        W = self.ctx.ct_words
        return self.ctx.decode(self.ctx.decrypt(ct_tensor[i * W:(i + 1) * W]), log_scale)

    def export(self, t, count):
        return self.ctx.export(t, 2 * count).reshape(count, 2, self.par.L, self.par.n)


def padded(X, d):
    Xp = np.zeros((X.shape[0], d))
    Xp[:, :X.shape[1]] = X
    return Xp


def test_tiny_rows_fullsize():
    """1,024 x 128-d at N=2^13: row layout, ct x pt then 7 rotate-and-sum steps
    (all 32 outputs bit-exact), and one diagonal block as a cross-check."""
    w = wl.WORKLOADS["tiny"]
    st = Setup(w, oracle_steps=sorted(set(wl.rotation_steps(w) + ckks.steps_for_bsgs(w.d, w.B))))
    extra = [r for r in ckks.steps_for_bsgs(w.d, w.B) if not st.ctx.has_key(r)]
    rand = [wl.key_randomness(w, r, st.par.primes, st.par.dnum) for r in extra]
    st.ctx.keygen(st.s, extra, np.stack([x[0] for x in rand]), np.stack([x[1] for x in rand]))
    X, _ = wl.candidate_rows(w)
    q = wl.query_vectors(w)[0]
    ct, ct_o = st.encrypt_query(q)
    S = st.par.slots
    slot_pts = ckks.pack_rows(X.astype(np.float64), S, w.d)
    coeffs = np.stack([ckks.encode(v, st.par.n, 40) for v in slot_pts])
    say(f"[tiny] row layout, {len(coeffs)} plaintexts")
    pts = st.ctx.encode_db_block_int(coeffs)
    PW = st.ctx.pt_words
    out = st.ctx.score_block(ct, [pts[i * PW:(i + 1) * PW] for i in range(len(coeffs))], w.d, 0)
    st.ctx.rotate_sum(out, len(coeffs), 1, int(np.log2(w.d)))
    got = st.export(out, len(coeffs))
    scores = []
    for i in range(len(coeffs)):
        ref = st.orc.rotate_sum(st.orc.mul_plain(ct_o, ckks.to_residues(coeffs[i], st.par.q)), 1,
                                int(np.log2(w.d)), st.keys)
        assert np.array_equal(got[i], ref), i
        scores.extend(st.decode(out, i, 80)[::w.d])
    Xd = X.astype(np.float64)
    assert np.max(np.abs(np.array(scores)[:w.rows] - Xd @ q)) < 1e-4
    # diagonal layout on the same rows
    say("[tiny] diagonal cross-check")
    c = ckks.layout_b_coeffs(Xd, st.par, w.d, w.B)
    blk = st.ctx.encode_db_block_int(c)
    o2 = st.ctx.score_block(ct, [blk], w.d, 1, w.B)
    pts_o = np.stack([ckks.to_residues(x, st.par.q) for x in c]).reshape(w.G, w.B, st.par.L, st.par.n)
    ref = st.orc.bsgs_block(st.orc.baby_rotations(ct_o, w.B, st.keys), pts_o, w.B, w.G, st.keys)
    assert np.array_equal(st.export(o2, 1)[0], ref)
    assert np.max(np.abs(st.decode(o2, 0, 80)[:w.rows] - Xd @ q)) < 1e-4


def _multi_block(w):
    """Every block of the level bit-exact against the oracle: all blocks enrolled from the
    oracle's integer encoding (the same plaintexts on both sides), scored in one call as
    bench.py launches it; then the same rows enrolled by the library's float encoder score
    within 1e-4 of float64 as well."""
    st = Setup(w)
    X, centers = wl.candidate_rows(w)
    q = wl.query_vectors(w, 1, centers)[0]
    qp = np.zeros(w.d)
    qp[:len(q)] = q
    ct, ct_o = st.encrypt_query(qp)
    S = st.par.slots
    blocks, coeffs = [], []
    for b in range(w.n_blocks):
        rows = X[b * S:(b + 1) * S]
        coeffs.append(ckks.layout_b_coeffs(padded(rows.astype(np.float64), w.d), st.par, w.d, w.B))
        blocks.append(st.ctx.encode_db_block_int(coeffs[-1]))
        say(f"[{w.name}] block {b}: {len(rows)} rows encoded by the oracle")
    say(f"[{w.name}] scoring {w.n_blocks} blocks (B={w.B}, G={w.G}) on the GPU")
    out = st.ctx.score_block(ct, blocks, w.d, 1, w.B)
    got = st.export(out, w.n_blocks)
    say(f"[{w.name}] oracle: {w.B - 1} baby rotations")
    qrot = st.orc.baby_rotations(ct_o, w.B, st.keys)
    for b in range(w.n_blocks):
        pts_o = np.stack([ckks.to_residues(x, st.par.q) for x in coeffs[b]]).reshape(w.G, w.B, st.par.L,
                                                                                    st.par.n)
        assert np.array_equal(got[b], st.orc.bsgs_block(qrot, pts_o, w.B, w.G, st.keys)), b
        say(f"[{w.name}] block {b} bit-exact")
    del blocks, coeffs
    fblocks = [st.ctx.encode_db_block(X[b * S:(b + 1) * S], w.d, 1, w.B) for b in range(w.n_blocks)]
    outs = {"oracle-encoded": out, "float-encoded": st.ctx.score_block(ct, fblocks, w.d, 1, w.B)}
    for name, o in outs.items():
        err = 0.0
        for b in range(w.n_blocks):
            rows = X[b * S:(b + 1) * S].astype(np.float64)
            z = st.decode(o, b, 80)
            err = max(err, float(np.max(np.abs(z[:len(rows)] - rows @ q))))
            if len(rows) < S:
                err = max(err, float(np.max(np.abs(z[len(rows):]))))
        say(f"[{w.name}] {name} blocks: max |score - float64| = {err:.2e}")
        assert err < 1e-4


def test_fine_level_fullsize():
    """65,536 x 96-d (zero-padded to 128) at N=2^15: 4 diagonal blocks, all bit-exact;
    every score is the exact 96-d cosine."""
    _multi_block(wl.WORKLOADS["fine"])


def test_rerank_level_fullsize():
    """110,000 x 512-d at N=2^16, B=64: 4 blocks as bench.py times them, all bit-exact (the
    last one partial, 11,696 rows); all 110,000 scores within 1e-4 of float64."""
    _multi_block(wl.WORKLOADS["rerank"])


def test_rank_reduction_fullsize():
    """Encrypted 512 -> 128 projection (hybrid diagonals, BSGS, one fold) then 16,384
    candidates at d=128; both ciphertexts bit-exact; norm-corrected cosines vs float64."""
    w = wl.WORKLOADS["rank"]
    st = Setup(w)
    W = wl.projection(w)
    q = wl.query_vectors(w)[0]
    ct, ct_o = st.encrypt_query(q)
    S = st.par.slots
    R, Bp = w.d, w.B_proj
    pre = ckks.prerotate(ckks.projection_diagonals(W, S), Bp)
    wco = np.stack([ckks.encode(pre[g, b], st.par.n, 40) for g in range(R // Bp) for b in range(Bp)])
    wpts = st.ctx.encode_db_block_int(wco)
    say("[rank] projection on the GPU")
    qr = st.ctx.project_ct(ct, wpts, w.d_in, R, Bp)
    Xr = wl.projected_rows(w, W)
    c = ckks.layout_b_coeffs(Xr, st.par, R, w.B)
    blk = st.ctx.encode_db_block_int(c)
    out = st.ctx.score_block(qr, [blk], R, 1, w.B)
    say("[rank] oracle projection + fold + scoring")
    wres = np.stack([ckks.to_residues(x, st.par.q) for x in wco]).reshape(R // Bp, Bp, st.par.L, st.par.n)
    z = st.orc.bsgs_block(st.orc.baby_rotations(ct_o, Bp, st.keys), wres, Bp, R // Bp, st.keys)
    z = st.orc.rotate_sum(z, R, int(np.log2(w.d_in // R)), st.keys)
    assert np.array_equal(st.export(qr, 1)[0], z)
    pts_o = np.stack([ckks.to_residues(x, st.par.q) for x in c]).reshape(w.G, w.B, st.par.L, st.par.n)
    ref = st.orc.bsgs_block(st.orc.baby_rotations(z, w.B, st.keys), pts_o, w.B, w.G, st.keys)
    assert np.array_equal(st.export(out, 1)[0], ref)
    qR = W.T @ q
    raw = st.decode(out, 0, 120)[:w.rows]
    cos = raw / np.linalg.norm(qR)
    assert np.max(np.abs(cos - Xr @ qR / np.linalg.norm(qR))) < 1e-4
    # W's diagonals encrypted (as bench.py times it): the projection decrypts to W^T q
    say("[rank] projection with W encrypted")
    ra, re_ = wl.relin_randomness(w, st.par.primes, st.par.dnum)
    st.ctx.keygen_relin(st.s, ra, re_)
    a, e = wl.db_enc_randomness(w, st.par.q, 0, R, block=99)
    wct = st.ctx.encrypt_pts(wpts, R, a, e)
    qr_e = st.ctx.project_ct_enc(ct, wct, w.d_in, R, Bp)
    assert np.max(np.abs(st.decode(qr_e, 0, 80) - np.tile(qR, S // R))) < 1e-4


def test_rerank_level_at_three_primes_fullsize():
    """Level drop: the query (encrypted at all 12 primes) is dropped to 3 ciphertext primes and
    the 110,000 x 512 rerank level is scored there, with the database enrolled at that level and
    the rotation keys restricted.  Dropped ciphertext, one rotation and the last block bit-exact
    against the oracle at the lower level; all scores within 1e-4."""
    from paper_2608_21131_amd import fa
    w = wl.WORKLOADS["rerank"]
    L_low = 3
    par = ckks.Params(logn=w.log_n, L=w.L, K=w.K)
    lp = ckks.Params(logn=w.log_n, L=L_low, K=w.K, primes=par.q[:L_low] + par.p)
    ctx = fa.Context(w.log_n, w.L, w.K, 40)
    s = wl.secret(w)
    steps = wl.rotation_steps(w)
    say(f"[low] keys for {len(steps)} rotations at 12 primes")
    for i in range(0, len(steps), 8):
        chunk = steps[i:i + 8]
        rand = [wl.key_randomness(w, r, par.primes, par.dnum) for r in chunk]
        ctx.keygen(s, chunk, np.stack([x[0] for x in rand]), np.stack([x[1] for x in rand]))
    low = ctx.at_level(L_low)
    assert low.primes == lp.primes
    lo = ckks.Oracle(lp)
    idx = list(range(L_low)) + list(range(par.L, par.L + par.K))
    keys = {}
    for r in steps:
        a, e = wl.key_randomness(w, r, par.primes, par.dnum)
        keys[r] = lo.keygen(s, r, a[:lp.dnum][:, idx], e[:lp.dnum])
    X, centers = wl.candidate_rows(w)
    q = wl.query_vectors(w, 1, centers)[0]
    a, e = wl.enc_randomness(w, par.q)
    m = ckks.encode(ckks.replicate(q, par.slots), par.n, 40)
    ct = ctx.encrypt(m, a, e)
    ct_low = ctx.drop_level(low, ct)
    full_o = ckks.Oracle(par).encrypt(m, a, e, s)
    ct_low_o = np.ascontiguousarray(full_o[:, :L_low])
    assert np.array_equal(low.export(ct_low, 2).reshape(2, L_low, par.n), ct_low_o)
    say("[low] one rotation at 3 primes")
    assert np.array_equal(low.export(low.rotate(ct_low, 5), 2).reshape(2, L_low, par.n),
                          lo.rotate(ct_low_o, 5, keys[5]))
    S = par.slots
    blocks, ref_coeffs = [], None
    for b in range(w.n_blocks):
        rows = X[b * S:(b + 1) * S]
        if b == w.n_blocks - 1:
            ref_coeffs = ckks.layout_b_coeffs(rows.astype(np.float64), lp, w.d, w.B)
            blocks.append(low.encode_db_block_int(ref_coeffs))
        else:
            blocks.append(low.encode_db_block(rows, w.d, 1, w.B))
    say("[low] scoring 4 blocks at 3 primes")
    out = low.score_block(ct_low, blocks, w.d, 1, w.B)
    got = low.export(out, 2 * w.n_blocks).reshape(w.n_blocks, 2, L_low, par.n)[-1]
    qrot = lo.baby_rotations(ct_low_o, w.B, keys)
    pts_o = np.stack([ckks.to_residues(x, lp.q) for x in ref_coeffs]).reshape(w.G, w.B, L_low, par.n)
    assert np.array_equal(got, lo.bsgs_block(qrot, pts_o, w.B, w.G, keys))
    err = 0.0
    W_ = low.ct_words
    for b in range(w.n_blocks):
        rows = X[b * S:(b + 1) * S].astype(np.float64)
        z = low.decode(low.decrypt(out[b * W_:(b + 1) * W_]), 80)
        err = max(err, float(np.max(np.abs(z[:len(rows)] - rows @ q))))
    say(f"[low] max |score - float64| = {err:.2e}")
    assert err < 1e-4


def test_rerank_query_batch_fullsize():
    """Cross-query batching at the rerank level's full size: 5 queries prepared together
    (fa_prepare_batch: a step's key switches issued for all five) and scored in two plaintext
    passes (four queries, then one) against the 4 resident blocks.  Every output ciphertext
    equals the single-query path word for word; the second query's last block (scored in the
    four-query pass) is bit-exact against the oracle; every decrypted score is within 1e-4 of
    float64."""
    w = wl.WORKLOADS["rerank"]
    st = Setup(w)
    X, centers = wl.candidate_rows(w)
    Q = wl.query_vectors(w, 5, centers)
    S = st.par.slots
    last = X[(w.n_blocks - 1) * S:]
    c_last = ckks.layout_b_coeffs(last.astype(np.float64), st.par, w.d, w.B)
    blocks = [st.ctx.encode_db_block(X[b * S:(b + 1) * S], w.d, 1, w.B) for b in range(w.n_blocks - 1)]
    blocks.append(st.ctx.encode_db_block_int(c_last))
    cts, cts_o = [], []
    for j, v in enumerate(Q):
        a, e = wl.enc_randomness(w, st.par.q, tag=j)
        m = ckks.encode(ckks.replicate(v, S), st.par.n, 40)
        cts.append(st.ctx.encrypt(m, a, e))
        cts_o.append(st.orc.encrypt(m, a, e, st.s) if j == 1 else None)
    say(f"[batch] {len(Q)} queries prepared together")
    preps = st.ctx.prepare_batch(cts, w.B)
    say(f"[batch] {len(Q)} queries x {w.n_blocks} blocks")
    outs = st.ctx.score_batch(cts, preps, blocks, w.d, w.B)
    err = 0.0
    for j in range(len(Q)):
        single = st.ctx.score_block(cts[j], blocks, w.d, 1, w.B)
        assert np.array_equal(st.export(outs[j], w.n_blocks), st.export(single, w.n_blocks)), j
        for b in range(w.n_blocks):
            rows = X[b * S:(b + 1) * S].astype(np.float64)
            z = st.decode(outs[j], b, 80)
            err = max(err, float(np.max(np.abs(z[:len(rows)] - rows @ Q[j]))))
    say(f"[batch] max |score - float64| = {err:.2e}; oracle: query 1's rotations and last block")
    assert err < 1e-4
    pts_o = np.stack([ckks.to_residues(x, st.par.q) for x in c_last]).reshape(w.G, w.B, st.par.L, st.par.n)
    ref = st.orc.bsgs_block(st.orc.baby_rotations(cts_o[1], w.B, st.keys), pts_o, w.B, w.G, st.keys)
    assert np.array_equal(st.export(outs[1], w.n_blocks)[-1], ref)


def test_three_level_fullsize_at_all_primes():
    """The full three-level query at its own parameters (N=2^16, 12+3 primes), as bench.py runs
    it: four queries prepared together and scored in one pass over the 7 coarse blocks
    (222,049 centroids); the client decrypts, keeps the top 16 and names 2 of the 4 fine-pool
    blocks by id; then the top 64 name 4 of the 8 rerank-pool blocks.  For the first query the
    last coarse block, the second fine block and the last rerank block are bit-exact against
    the oracle; every score of every level is within 1e-4 of float64."""
    w = wl.WORKLOADS["three_level"]
    ex = w.extra
    st = Setup(w)
    S = st.par.slots
    coarse, centers = wl.candidate_rows(w, ex["coarse"], stream_extra=1)
    pools, rows_of, ref_coeffs = {}, {}, {}
    n_coarse = -(-ex["coarse"] // S)
    rows_of["coarse"] = [coarse[b * S:(b + 1) * S] for b in range(n_coarse)]
    for name, nb, extra in (("fine", ex["fine_pool_blocks"], 2), ("rerank", ex["rerank_pool_blocks"], 3)):
        X, _ = wl.candidate_rows(w, nb * S, stream_extra=extra, centers=centers)
        rows_of[name] = [X[b * S:(b + 1) * S] for b in range(nb)]
    # the rerank level's last block is truncated like bench.py's (11,696 rows)
    Q = wl.query_vectors(w, 4, centers)
    # blocks a check may select are enrolled from the oracle's integer encoding (the same
    # plaintexts on both sides); the other coarse blocks by the library's float encoder
    for name in ("coarse", "fine", "rerank"):
        pools[name] = []
        for b, r in enumerate(rows_of[name]):
            if name == "coarse" and b < n_coarse - 1:
                pools[name].append(st.ctx.encode_db_block(r, w.d, 1, w.B))
                continue
            ref_coeffs[(name, b)] = ckks.layout_b_coeffs(r.astype(np.float64), st.par, w.d, w.B)
            pools[name].append(st.ctx.encode_db_block_int(ref_coeffs[(name, b)]))
        say(f"[3lvl-12] {name}: {len(pools[name])} resident blocks at 12 primes")
    cts, q0_o = [], None
    for j, v in enumerate(Q):
        a, e = wl.enc_randomness(w, st.par.q, tag=j)
        m = ckks.encode(ckks.replicate(v, S), st.par.n, 40)
        cts.append(st.ctx.encrypt(m, a, e))
        if j == 0:
            q0_o = st.orc.encrypt(m, a, e, st.s)

    def scores(out, nb, rows_list, qv, n_last=None):
        zs, err = [], 0.0
        for b in range(nb):
            n_valid = len(rows_list[b]) if (b < nb - 1 or n_last is None) else n_last
            z = st.decode(out, b, 80)[:n_valid]
            err = max(err, float(np.max(np.abs(z - rows_list[b][:n_valid].astype(np.float64) @ qv))))
            zs.append(z)
        return np.concatenate(zs), err

    def top(sc, k):
        return np.lexsort((np.arange(len(sc)), -sc))[:k]

    say("[3lvl-12] coarse: 4 queries prepared and scored in one pass")
    preps = st.ctx.prepare_batch(cts, w.B)
    outs_c = st.ctx.score_batch(cts, preps, pools["coarse"], w.d, w.B)
    checks = {}
    errs = []
    for j in range(len(Q)):
        sc, err = scores(outs_c[j], n_coarse, rows_of["coarse"], Q[j])
        errs.append(err)
        fsel = sorted(set(int(x) % ex["fine_pool_blocks"] for x in top(sc, ex["top_coarse"])))
        fsel = (fsel + [b for b in range(ex["fine_pool_blocks"]) if b not in fsel])[:ex["fine_blocks"]]
        out_f = st.ctx.score_prepared(cts[j], preps[j], pools["fine"], w.d, w.B, block_ids=fsel)
        fr = [rows_of["fine"][b] for b in fsel]
        sc, err = scores(out_f, len(fsel), fr, Q[j])
        errs.append(err)
        rsel = sorted(set(int(x) % ex["rerank_pool_blocks"] for x in top(sc, ex["top_fine"])))
        rsel = (rsel + [b for b in range(ex["rerank_pool_blocks"]) if b not in rsel])[:ex["rerank_blocks"]]
        out_r = st.ctx.score_prepared(cts[j], preps[j], pools["rerank"], w.d, w.B, block_ids=rsel)
        rr = [rows_of["rerank"][b] for b in rsel]
        _, err = scores(out_r, len(rsel), rr, Q[j], n_last=ex["rerank_last"])
        errs.append(err)
        if j == 0:
            checks = {"coarse": (outs_c[0], n_coarse - 1, ("coarse", n_coarse - 1)),
                      "fine": (out_f, len(fsel) - 1, ("fine", fsel[-1])),
                      "rerank": (out_r, len(rsel) - 1, ("rerank", rsel[-1]))}
        say(f"[3lvl-12] query {j}: fine blocks {fsel}, rerank blocks {rsel}")
    say(f"[3lvl-12] max |score - float64| = {max(errs):.2e}")
    assert max(errs) < 1e-4
    say("[3lvl-12] oracle: the first query's baby rotations")
    qrot = st.orc.baby_rotations(q0_o, w.B, st.keys)
    for name, (out, b, key) in checks.items():
        c = ref_coeffs[key]
        pts_o = np.stack([ckks.to_residues(x, st.par.q) for x in c]).reshape(w.G, w.B, st.par.L, st.par.n)
        got = st.export(out, b + 1)[b]
        say(f"[3lvl-12] oracle: {name} block {b}")
        assert np.array_equal(got, st.orc.bsgs_block(qrot, pts_o, w.B, w.G, st.keys)), name


def test_three_level_coarse_batch_at_three_primes_fullsize():
    """The full three-level query's coarse level as bench.py runs it: 222,049 x 512-d centroids
    in 7 blocks enrolled at 3 primes, four queries dropped to 3 primes, prepared together
    (fa_prepare_batch) and scored in one plaintext pass (fa_score_batch).  The first query's
    last, partial block bit-exact against the oracle at the lower level; every score of the
    four queries within 1e-4 of float64."""
    from paper_2608_21131_amd import fa
    w = wl.WORKLOADS["three_level"]
    ex = w.extra
    L_low = 3
    par = ckks.Params(logn=w.log_n, L=w.L, K=w.K)
    lp = ckks.Params(logn=w.log_n, L=L_low, K=w.K, primes=par.q[:L_low] + par.p)
    ctx = fa.Context(w.log_n, w.L, w.K, 40)
    s = wl.secret(w)
    steps = wl.rotation_steps(w)
    say(f"[3lvl] keys for {len(steps)} rotations")
    for i in range(0, len(steps), 8):
        chunk = steps[i:i + 8]
        rand = [wl.key_randomness(w, r, par.primes, par.dnum) for r in chunk]
        ctx.keygen(s, chunk, np.stack([x[0] for x in rand]), np.stack([x[1] for x in rand]))
    low = ctx.at_level(L_low)
    lo = ckks.Oracle(lp)
    idx = list(range(L_low)) + list(range(par.L, par.L + par.K))
    keys = {}
    for r in ckks.steps_for_bsgs(w.d, w.B):
        a, e = wl.key_randomness(w, r, par.primes, par.dnum)
        keys[r] = lo.keygen(s, r, a[:lp.dnum][:, idx], e[:lp.dnum])
    X, centers = wl.candidate_rows(w, ex["coarse"], stream_extra=1)
    S = par.slots
    nb = -(-ex["coarse"] // S)
    blocks, ref_coeffs = [], None
    for b in range(nb):
        rows = X[b * S:(b + 1) * S]
        if b == nb - 1:
            ref_coeffs = ckks.layout_b_coeffs(rows.astype(np.float64), lp, w.d, w.B)
            blocks.append(low.encode_db_block_int(ref_coeffs))
        else:
            blocks.append(low.encode_db_block(rows, w.d, 1, w.B))
    Q = wl.query_vectors(w, 4, centers)
    full_o = ckks.Oracle(par)
    qs, q0_o = [], None
    for j, v in enumerate(Q):
        a, e = wl.enc_randomness(w, par.q, tag=j)
        m = ckks.encode(ckks.replicate(v, S), par.n, 40)
        qs.append(ctx.drop_level(low, ctx.encrypt(m, a, e)))
        if j == 0:
            q0_o = np.ascontiguousarray(full_o.encrypt(m, a, e, s)[:, :L_low])
    say(f"[3lvl] 4 queries x {nb} coarse blocks at {L_low} primes, prepared and scored together")
    preps = low.prepare_batch(qs, w.B)
    outs = low.score_batch(qs, preps, blocks, w.d, w.B)
    got = low.export(outs[0], 2 * nb).reshape(nb, 2, L_low, par.n)[-1]
    say("[3lvl] oracle: baby rotations + the last block for the first query")
    pts_o = np.stack([ckks.to_residues(x, lp.q) for x in ref_coeffs]).reshape(w.G, w.B, L_low, par.n)
    assert np.array_equal(got, lo.bsgs_block(lo.baby_rotations(q0_o, w.B, keys), pts_o, w.B, w.G, keys))
    err = 0.0
    W_ = low.ct_words
    for j in range(len(Q)):
        for b in range(nb):
            rows = X[b * S:(b + 1) * S].astype(np.float64)
            z = low.decode(low.decrypt(outs[j][b * W_:(b + 1) * W_]), 80)
            err = max(err, float(np.max(np.abs(z[:len(rows)] - rows @ Q[j]))))
            if len(rows) < S:
                err = max(err, float(np.max(np.abs(z[len(rows):]))))
    say(f"[3lvl] max |score - float64| = {err:.2e}")
    assert err < 1e-4


def test_rerank_encrypted_database_at_three_primes_fullsize():
    """The rerank level against an encrypted database (every diagonal a ciphertext, enrolled at
    3 primes), ct x ct with one relinearisation per (block, giant): the last block's output
    and its encrypted diagonals bit-exact against the oracle at the lower level; all 110,000
    scores within 1e-4 of float64."""
    from paper_2608_21131_amd import fa
    w = wl.WORKLOADS["rerank"]
    L_low = 3
    par = ckks.Params(logn=w.log_n, L=w.L, K=w.K)
    lp = ckks.Params(logn=w.log_n, L=L_low, K=w.K, primes=par.q[:L_low] + par.p)
    ctx = fa.Context(w.log_n, w.L, w.K, 40)
    s = wl.secret(w)
    steps = wl.rotation_steps(w)
    say(f"[enc] keys for {len(steps)} rotations + relinearisation at 12 primes")
    for i in range(0, len(steps), 8):
        chunk = steps[i:i + 8]
        rand = [wl.key_randomness(w, r, par.primes, par.dnum) for r in chunk]
        ctx.keygen(s, chunk, np.stack([x[0] for x in rand]), np.stack([x[1] for x in rand]))
    ra, re_ = wl.relin_randomness(w, par.primes, par.dnum)
    ctx.keygen_relin(s, ra, re_)
    low = ctx.at_level(L_low)
    assert low.has_relin_key()
    lo = ckks.Oracle(lp)
    idx = list(range(L_low)) + list(range(par.L, par.L + par.K))
    keys = {}
    for r in steps:
        a, e = wl.key_randomness(w, r, par.primes, par.dnum)
        keys[r] = lo.keygen(s, r, a[:lp.dnum][:, idx], e[:lp.dnum])
    rlk = lo.keygen_relin(s, ra[:lp.dnum][:, idx], re_[:lp.dnum])
    X, centers = wl.candidate_rows(w)
    q = wl.query_vectors(w, 1, centers)[0]
    a, e = wl.enc_randomness(w, par.q)
    m = ckks.encode(ckks.replicate(q, par.slots), par.n, 40)
    ct_low = ctx.drop_level(low, ctx.encrypt(m, a, e))
    ct_low_o = np.ascontiguousarray(ckks.Oracle(par).encrypt(m, a, e, s)[:, :L_low])
    S = par.slots
    blocks = []
    last_o = None
    for b in range(w.n_blocks):
        rows = X[b * S:(b + 1) * S]
        ea, ee = wl.db_enc_randomness(w, lp.q, 0, w.d, block=b)
        if b == w.n_blocks - 1:
            c = ckks.layout_b_coeffs(rows.astype(np.float64), lp, w.d, w.B)
            cts = low.encrypt_pts(low.encode_db_block_int(c), w.d, ea, ee)
            say("[enc] oracle encryption of the last block")
            last_o = np.stack([lo.encrypt(c[j], ea[j], ee[j], s) for j in range(w.d)])
            assert np.array_equal(low.export(cts, 2 * w.d).reshape(w.d, 2, L_low, par.n), last_o)
        else:
            cts = low.encrypt_pts(low.encode_db_block(rows, w.d, 1, w.B), w.d, ea, ee)
        blocks.append(cts)
    say("[enc] scoring 4 encrypted blocks at 3 primes")
    out = low.score_block(ct_low, blocks, w.d, fa.LAYOUT_DIAG_ENC, w.B)
    got = low.export(out, 2 * w.n_blocks).reshape(w.n_blocks, 2, L_low, par.n)[-1]
    say("[enc] oracle: baby rotations + encrypted last block")
    qrot = lo.baby_rotations(ct_low_o, w.B, keys)
    ref = lo.bsgs_block_ct(qrot, last_o.reshape(w.G, w.B, 2, L_low, par.n), w.B, w.G, keys, rlk)
    assert np.array_equal(got, ref)
    err = 0.0
    W_ = low.ct_words
    for b in range(w.n_blocks):
        rows = X[b * S:(b + 1) * S].astype(np.float64)
        z = low.decode(low.decrypt(out[b * W_:(b + 1) * W_]), 80)
        err = max(err, float(np.max(np.abs(z[:len(rows)] - rows @ q))))
    say(f"[enc] max |score - float64| = {err:.2e}")
    assert err < 1e-4


def test_membership_face_scan_fullsize():
    """The face membership scan at full size, as bench.py times it: an encrypted 512-d query
    (scale 2^50, 12 primes) projected to R = 128 and rescaled, then 222,049 centroids in 7
    blocks at 11 primes, tau |q_R| by the degree-7 Chebyshev series and two sign steps
    (levels 12 -> 2).  The projected query and the ragged last block's output are bit-exact
    against the oracle; every output is within 1e-4 of the float64 model, every decision
    whose margin exceeds the series' error is cos >= tau, and the query's own identity is
    the one match."""
    from paper_2608_21131_amd import fa
    w = wl.WORKLOADS["face"]
    x = w.extra
    top = ckks.Params(logn=w.log_n, L=w.L, K=w.K, log_scale=x["log_scale"])
    S, R, B, Bp = top.slots, w.d, w.B, w.B_proj
    ctx = fa.Context(w.log_n, w.L, w.K, x["log_scale"])
    assert ctx.primes == top.primes
    s = wl.secret(w)
    steps = wl.rotation_steps(w)
    rlk = wl.relin_randomness(w, top.primes, top.dnum)
    rot = {r: wl.key_randomness(w, r, top.primes, top.dnum) for r in steps}
    say(f"[face] keys: relinearisation + {len(steps)} rotations, then levels 11..2")
    ctx.keygen_relin(s, *rlk)
    for i in range(0, len(steps), 8):
        chunk = steps[i:i + 8]
        ctx.keygen(s, chunk, np.stack([rot[r][0] for r in chunk]), np.stack([rot[r][1] for r in chunk]))
    levels = [ctx] + [ctx.at_level(l) for l in range(w.L - 1, 1, -1)]
    W = wl.projection(w)
    qs, ids = wl.face_queries(w)
    q, ident = qs[0], int(ids[0])
    m = ckks.encode(ckks.replicate(q, S), top.n, x["log_scale"])
    a, e = wl.enc_randomness(w, top.q)
    ct = ctx.encrypt(m, a, e)
    pre = ckks.prerotate(ckks.projection_diagonals(W, S), Bp)
    wco = np.stack([ckks.encode(pre[g, b], top.n, x["log_scale"]) for g in range(R // Bp) for b in range(Bp)])
    say("[face] projection and rescale on the GPU")
    qr = ctx.project_ct(ct, ctx.encode_db_block_int(wco), w.d_in, R, Bp)
    q11 = ctx.rescale(levels[1], qr)
    s_q = 2.0 ** (2 * x["log_scale"]) / top.q[-1]
    Xr = wl.projected_rows(w, W)
    nb = w.n_blocks
    lp = ckks.Params(logn=w.log_n, L=w.L - 1, K=w.K, log_scale=x["log_scale"], primes=top.q[:w.L - 1] + top.p)
    last = Xr[(nb - 1) * S:]
    blocks = [levels[1].encode_db_block(Xr[i * S:(i + 1) * S].astype(np.float32), R, fa.LAYOUT_DIAG, B)
              for i in range(nb - 1)]
    blocks.append(levels[1].encode_db_block_int(ckks.layout_b_coeffs(last, lp, R, B)))
    coeffs = fa.cheb_fit_sqrt(x["tau"], x["y_lo"], x["y_hi"], x["degree"])
    say(f"[face] membership scan over {nb} blocks")
    out, L, sc, mo = fa.membership(levels, q11, w.L - 1, s_q, blocks, R, B, x["y_lo"], x["y_hi"], coeffs,
                                   x["m"], x["iters"])
    assert L == 2
    # float64 model and decisions over all 222,049 centroids
    ctw = levels[1].ct_words
    c2 = levels[w.L - L]
    at_L = [c2.wrap(out.t[i * ctw:i * ctw + 2 * L * c2.n], 2, 1, 0) for i in range(nb)]
    z = np.concatenate([c2.decode(c2.decrypt(b_), 50) for b_ in at_L])
    z = z[:w.rows] * (2.0 ** 50 / sc) / mo
    qR = W.T @ q
    Xm = np.vstack([Xr[:(nb - 1) * S].astype(np.float32).astype(np.float64), last])
    y = float(qR @ qR)
    assert x["y_lo"] < y < x["y_hi"]
    u = (2 * y - x["y_lo"] - x["y_hi"]) / (x["y_hi"] - x["y_lo"])
    t = np.polynomial.chebyshev.chebval(u, coeffs)
    err = abs(t - x["tau"] * np.sqrt(y))
    v = (Xm @ qR - t) / x["m"]
    for _ in range(x["iters"]):
        v = (3 * v - v ** 3) / 2
    assert np.max(np.abs(z - v)) < 1e-4
    margin = Xm @ qR - x["tau"] * np.sqrt(y)
    ok = np.abs(margin) > err + 1e-4
    assert np.all(np.sign(z[ok]) == np.sign(margin[ok]))
    assert np.flatnonzero(z > 0).tolist() == [ident]
    say(f"[face] y={y:.4f} series error {err:.2e}; identity {ident} matched; oracle chain")
    # oracle: the projection, its rescale, and the last block's scan
    ch = ckks.LevelChain(top, s, rlk, rot, rot_levels=[w.L, w.L - 1, w.L - 2])
    ct_o = ch.orc[w.L].encrypt(m, a, e, s)
    keys = ch.keys[w.L]
    wres = np.stack([ckks.to_residues(v_, top.q) for v_ in wco]).reshape(R // Bp, Bp, w.L, top.n)
    zo = ch.orc[w.L].bsgs_block(ch.orc[w.L].baby_rotations(ct_o, Bp, keys), wres, Bp, R // Bp, keys)
    zo = ch.orc[w.L].rotate_sum(zo, R, int(np.log2(w.d_in // R)), keys)
    assert np.array_equal(ctx.export(qr, 2).reshape(2, w.L, top.n), zo)
    q11o = ch.orc[w.L].rescale(zo)
    assert np.array_equal(levels[1].export(q11, 2).reshape(2, w.L - 1, top.n), q11o)
    say("[face] oracle scan of the last block")
    oo, Lo, so, mo2 = ckks.membership(ch, q11o, w.L - 1, s_q, [ckks.layout_b_pts(last, lp, R, B)], R, B,
                                      x["y_lo"], x["y_hi"], coeffs, x["m"], x["iters"])
    assert (Lo, so, mo2) == (L, sc, mo)
    assert np.array_equal(c2.export(at_L[nb - 1], 2).reshape(2, L, top.n), oo[0])
