"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Ciphertexts are compared word for word in canonical coefficient form
(bit-exact); decrypted scores against float64 inner products (<= 1e-4)."""
import numpy as np
import pytest

from oracle import ckks
from paper_2608_21131_amd import gen

from common import Pair, say

pytestmark = pytest.mark.gpu

_PAIRS = {}


def pair(name, wid=0):
    key = (name, wid)
    if key not in _PAIRS:
        say(f"[setup] context {name} wid={wid}")
        _PAIRS[key] = Pair(name, wid)
    return _PAIRS[key]


def rand_coeffs(g, n, count, bits=62):
    return g.integers(-(1 << bits), 1 << bits, size=(count, n), dtype=np.int64)


@pytest.mark.parametrize("name", ["tiny", "p1", "p2", "p4"])
def test_ntt_roundtrip_and_residues(name):
    p = pair(name)
    g = np.random.default_rng(1)
    c = rand_coeffs(g, p.n, 3)
    say(f"[ntt] {name} encode_db_block_int + export")
    pts = p.ctx.encode_db_block_int(c)
    got = p.ctx.export(pts, 3)
    for i in range(3):
        assert np.array_equal(got[i], ckks.to_residues(c[i], p.par.q)), i


@pytest.mark.parametrize("name", ["tiny", "p1", "p2", "p4"])
def test_encrypt_decrypt_parity(name):
    p = pair(name)
    v = np.random.default_rng(2).uniform(-1, 1, p.par.slots)
    m = ckks.encode(v, p.n, 40)
    say(f"[enc] {name}")
    ct_dev, ct_orc = p.encrypt_both(m)
    assert np.array_equal(p.export_ct(ct_dev)[0], ct_orc)
    res = p.ctx.decrypt(ct_dev)
    assert np.array_equal(res, p.orc.decrypt(ct_orc, p.s))
    z = p.ctx.decode(res, 40)
    assert np.max(np.abs(z - v)) < 1e-6


@pytest.mark.parametrize("name,steps", [("tiny", [1, 3, 100]), ("tiny1", [1, 5]), ("small", [1, 7]),
                                        ("p1", [1, 64]), ("p2", [5]), ("p4", [1]), ("s12", [1, 9]),
                                        ("s14", [1, 33]), ("d8", [1, 17]), ("max8", [1, 12345]),
                                        ("max20", [3])])
def test_rotation_parity(name, steps):
    p = pair(name)
    v = np.random.default_rng(3).uniform(-1, 1, p.par.slots)
    ct_dev, ct_orc = p.encrypt_both(ckks.encode(v, p.n, 40), tag=3)
    keys = p.keys(steps)
    for r in steps:
        say(f"[rot] {name} step {r}")
        got = p.export_ct(p.ctx.rotate(ct_dev, r))[0]
        ref = p.orc.rotate(ct_orc, r, keys[r])
        assert np.array_equal(got, ref), r
        # key-switch noise grows with N (the extended digits are not centred):
        # about 1e-6 at N = 2^13 and 3e-5 at N = 2^16, identical in the oracle
        z = p.ctx.decode(p.ctx.decrypt(p.ctx.rotate(ct_dev, r)), 40)
        assert np.max(np.abs(z - np.roll(v, -r))) < 1e-4


@pytest.mark.parametrize("name,d,rows", [("tiny", 16, 500), ("p1", 128, 1024)])
def test_row_layout_then_rotate_sum(name, d, rows):
    """Row-packed scoring: ct x pt per plaintext, then log2(d) rotate-and-sum steps."""
    p = pair(name, wid=4)
    X = gen.gaussian_unit_rows(gen.rng(4, gen.STREAM_DB), rows, d)
    q = gen.gaussian_unit_rows(gen.rng(4, gen.STREAM_QUERY), 1, d)[0]
    S = p.par.slots
    ct_dev, ct_orc = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=4)
    slot_pts = ckks.pack_rows(X, S, d)
    coeffs = np.stack([ckks.encode(v, p.n, 40) for v in slot_pts])
    steps = int(np.log2(d))
    keys = p.keys([1 << k for k in range(steps)])
    say(f"[rowA] {name} d={d} rows={rows} pts={len(coeffs)}")
    pts = p.ctx.encode_db_block_int(coeffs)
    W = p.ctx.pt_words
    blocks = [pts[w * W:(w + 1) * W] for w in range(len(coeffs))]
    out = p.ctx.score_block(ct_dev, blocks, d, 0)
    p.ctx.rotate_sum(out, len(coeffs), 1, steps)
    got = p.export_ct(out, len(coeffs))
    scores = []
    for w in range(len(coeffs)):
        pt_res = ckks.to_residues(coeffs[w], p.par.q)
        ref = p.orc.rotate_sum(p.orc.mul_plain(ct_orc, pt_res), 1, steps, keys)
        assert np.array_equal(got[w], ref), w
        z = p.ctx.decode(p.ctx.decrypt(out[w * p.ctx.ct_words:(w + 1) * p.ctx.ct_words]), 80)
        scores.extend(z[::d])
    assert np.max(np.abs(np.array(scores)[:rows] - X @ q)) < 1e-4


@pytest.mark.parametrize("name,d,B,rows_list", [
    ("tiny", 16, 4, [300, 512, 17]),
    ("tiny", 16, 1, [100]),
    ("tiny", 16, 16, [100]),
    ("tiny", 512, 8, [300]),    # d = N/2 (the widest block), G = 64 > 32 giants per giant-kernel launch
    ("tiny", 512, 64, [512]),   # d = N/2 with a full block of rows
    ("tiny", 16, 4, [512] * 16 + [5]),  # 17 blocks: the giant steps in two chunks of blocks
    ("tiny", 16, 4, [64] * 33),          # 33 blocks: more than one multiply-accumulate launch holds
    ("tiny1", 16, 4, [300, 512]),        # one digit: the fused special-prime kernel
    ("tiny1", 64, 8, [512]),
    ("p1", 128, 16, [4096, 1000]),
    ("p2", 128, 16, [3000]),
    ("s12", 64, 8, [700, 2048]),         # short last digit, N = 2^12
    ("s14", 128, 16, [5000]),            # short last digit with four-prime digits, N = 2^14
    ("d8", 64, 8, [1500]),               # eight key-switch digits
    ("max8", 16, 4, [32768, 3000]),      # eight digits of 16 primes at N = 2^16
])
def test_diag_score_parity(name, d, B, rows_list):
    p = pair(name, wid=5)
    S = p.par.slots
    G = d // B
    g = gen.rng(5, gen.STREAM_DB, d, B)
    Xs = [gen.gaussian_unit_rows(g, r, d) for r in rows_list]
    q = gen.gaussian_unit_rows(gen.rng(5, gen.STREAM_QUERY), 1, d)[0]
    ct_dev, ct_orc = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=5)
    keys = p.keys(ckks.steps_for_bsgs(d, B))
    blocks = []
    coeffs = []
    for X in Xs:
        c = ckks.layout_b_coeffs(X, p.par, d, B)
        coeffs.append(c)
        blocks.append(p.ctx.encode_db_block_int(c))
    say(f"[diag] {name} d={d} B={B} blocks={rows_list}")
    out = p.ctx.score_block(ct_dev, blocks, d, 1, B)
    got = p.export_ct(out, len(Xs))
    qrot = p.orc.baby_rotations(ct_orc, B, keys)
    for i, (X, c) in enumerate(zip(Xs, coeffs)):
        pts = np.stack([ckks.to_residues(ci, p.par.q) for ci in c]).reshape(G, B, p.par.L, p.n)
        ref = p.orc.bsgs_block(qrot, pts, B, G, keys)
        assert np.array_equal(got[i], ref), i
        z = p.ctx.decode(p.ctx.decrypt(out[i * p.ctx.ct_words:(i + 1) * p.ctx.ct_words]), 80)
        assert np.max(np.abs(z[:len(X)] - X @ q)) < 1e-4
        if len(X) < S:
            assert np.max(np.abs(z[len(X):])) < 1e-4


@pytest.mark.parametrize("name,d_in,R,B,rows", [
    ("small", 64, 16, 4, 100),
    ("small", 16, 16, 4, 100),   # R = d_in: no fold
    ("small", 64, 16, 1, 100),   # B = 1: no baby rotations
    ("p2", 512, 128, 16, 2000),
])
def test_projection_parity(name, d_in, R, B, rows):
    p = pair(name, wid=6)
    S = p.par.slots
    W = gen.projection_matrix(gen.rng(6, gen.STREAM_W), d_in, R, var=1.0 / R)
    q = gen.gaussian_unit_rows(gen.rng(6, gen.STREAM_QUERY), 1, d_in)[0]
    ct_dev, ct_orc = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=6)
    c = d_in // R
    fold = [R << k for k in range(int(np.log2(c)))]
    keys = p.keys(ckks.steps_for_bsgs(R, B) + fold)
    pre = ckks.prerotate(ckks.projection_diagonals(W, S), B)
    wco = np.stack([ckks.encode(pre[g, b], p.n, 40) for g in range(R // B) for b in range(B)])
    wpts = p.ctx.encode_db_block_int(wco)
    say(f"[proj] {name} d_in={d_in} R={R} B={B}")
    qr = p.ctx.project_ct(ct_dev, wpts, d_in, R, B)
    got = p.export_ct(qr)[0]
    wres = np.stack([ckks.to_residues(x, p.par.q) for x in wco]).reshape(R // B, B, p.par.L, p.n)
    z = p.orc.bsgs_block(p.orc.baby_rotations(ct_orc, B, keys), wres, B, R // B, keys)
    z = p.orc.rotate_sum(z, R, len(fold), keys)
    assert np.array_equal(got, z)
    qR = W.T @ q
    zz = p.ctx.decode(p.ctx.decrypt(qr), 80)
    assert np.max(np.abs(zz - np.tile(qR, S // R))) < 1e-4
    # score the projected query (scale 2^120) against normalised projected rows
    Xr = gen.normalize_rows(gen.gaussian_unit_rows(gen.rng(6, gen.STREAM_DB), rows, d_in) @ W)
    blk = p.ctx.encode_db_block(Xr.astype(np.float32), R, 1, B)
    out = p.ctx.score_block(qr, [blk], R, 1, B)
    raw = p.ctx.decode(p.ctx.decrypt(out), 120)[:rows]
    cos = raw / np.linalg.norm(qR)
    ref = Xr.astype(np.float32).astype(np.float64) @ qR / np.linalg.norm(qR)
    assert np.max(np.abs(cos - ref)) < 1e-4


@pytest.mark.parametrize("name,extra", [("p1", 0), ("p1", 40), ("p2", 40), ("p4", 40), ("p4", 80)])
def test_decode_matches_oracle_decode(name, extra):
    """The client decode (centred CRT over just enough primes, then the slot
    transform) against the oracle's big-integer CRT and numpy FFT, on the
    residues of m * 2^extra + noise for a slot vector encoded at 2^40: two
    primes at scale 2^40, three at 2^80 and 2^120; also a short n_slots."""
    p = pair(name)
    g = np.random.default_rng(11 + extra)
    v = g.uniform(-1, 1, p.par.slots)
    m = [int(x) * (1 << extra) + int(e) for x, e in zip(ckks.encode(v, p.n, 40), g.integers(-999, 999, p.n))]
    res = np.stack([np.array([x % q for x in m], dtype=np.uint64) for q in p.par.q])
    ls = 40 + extra
    say(f"[decode] {name} at 2^{ls}")
    got = p.ctx.decode(res, ls)
    ref = ckks.decode_residues(res, p.par, ls)
    assert np.max(np.abs(got - ref)) < 1e-12
    assert np.max(np.abs(got - v)) < 1e-6
    short = p.ctx.decode(res, ls, n_slots=37)
    assert short.shape == (37,) and np.array_equal(short, got[:37])


def test_save_and_load_enrolled_blocks(tmp_path):
    """save_buffers / load_buffers (fa_export_coeffs, then fa_import_coeffs): an enrolled block
    and a ciphertext come back word for word and score identically; a file saved for another
    ring is refused, and so is a residue that is not below its prime."""
    import torch
    from paper_2608_21131_amd import fa
    p = pair("p1", wid=19)
    S, d, B = p.par.slots, 128, 16
    p.keys(ckks.steps_for_bsgs(d, B), oracle=False)
    X = gen.gaussian_unit_rows(gen.rng(19, gen.STREAM_DB), 1000, d)
    q = gen.gaussian_unit_rows(gen.rng(19, gen.STREAM_QUERY), 1, d)[0]
    ct, _ = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=19)
    blk = p.ctx.encode_db_block(X.astype(np.float32), d, 1, B)
    path = str(tmp_path / "enrolled.npz")
    say("[save/load] p1")
    p.ctx.save_buffers(path, {"block": blk, "query": ct})
    got = p.ctx.load_buffers(path)
    assert torch.equal(got["block"].t, blk.t) and torch.equal(got["query"].t, ct.t)
    assert (got["block"].count, got["block"].n_polys, got["block"].log_scale) == (d, 1, 40)
    assert (got["query"].count, got["query"].n_polys, got["query"].log_scale) == (1, 2, 40)
    ref = p.export_ct(p.ctx.score_block(ct, [blk], d, 1, B))
    assert np.array_equal(p.export_ct(p.ctx.score_block(got["query"], [got["block"]], d, 1, B)), ref)
    with pytest.raises(ValueError):
        pair("tiny").ctx.load_buffers(path)
    bad = p.ctx.export(blk.item(0))
    bad[0, 1, 5] = p.par.q[1]
    with pytest.raises(fa.FaError, match="FA_E_INVAL"):
        p.ctx.import_coeffs(bad)


@pytest.mark.parametrize("name", ["tiny", "p4"])
def test_float_encode_matches_oracle(name):
    p = pair(name)
    v = np.random.default_rng(7).standard_normal(p.par.slots) * 0.1
    mine = p.ctx.encode(v, 40)
    ref = ckks.encode(v, p.n, 40)
    diff = np.abs(mine - ref)
    assert diff.max() <= 1
    assert np.count_nonzero(diff) <= max(2, p.n // 1000)


def test_encode_db_block_float_vs_oracle():
    p = pair("p1", wid=8)
    d, B = 128, 16
    X = gen.gaussian_unit_rows(gen.rng(8, gen.STREAM_DB), 3000, d).astype(np.float32)
    say("[encode_db_block] p1")
    pts = p.ctx.encode_db_block(X, d, 1, B)
    got = p.ctx.export(pts, d)
    ref = ckks.layout_b_coeffs(X.astype(np.float64), p.par, d, B)
    mism = 0
    for j in range(d):
        r = ckks.to_residues(ref[j], p.par.q)
        dif = (got[j].astype(np.int64) - r.astype(np.int64))
        qs = np.array(p.par.q, dtype=np.int64)[:, None]
        dif = np.where(dif > qs // 2, dif - qs, np.where(dif < -(qs // 2), dif + qs, dif))
        assert np.abs(dif).max() <= 1
        mism += int(np.count_nonzero(dif[0]))
    assert mism <= d * p.n // 1000
    say(f"[encode_db_block] coefficient mismatches (|dm| = 1): {mism} of {d * p.n}")


def test_error_paths():
    from paper_2608_21131_amd import fa
    p = pair("tiny", wid=9)
    ct = p.ctx.new_ct()
    ct.zero_()
    # missing rotation key
    with pytest.raises(fa.FaError) as ei:
        p.ctx.rotate(ct, 77)
    assert ei.value.code == fa.FA_E_NOKEY
    # workspace too small
    blk = p.ctx.new_pt(16)
    p.keys(ckks.steps_for_bsgs(16, 4), oracle=False)
    small = p.ctx.new_pt(1)
    with pytest.raises(fa.FaError) as ei:
        p.ctx.score_block(ct, [blk], 16, 1, 4, ws=small)
    assert ei.value.code == fa.FA_E_NOMEM
    # d not a power of two / baby step not dividing d
    with pytest.raises(fa.FaError) as ei:
        p.ctx.score_block(ct, [blk], 12, 1, 4)
    assert ei.value.code == fa.FA_E_SHAPE
    with pytest.raises(fa.FaError) as ei:
        p.ctx.score_block(ct, [blk], 16, 1, 3)
    assert ei.value.code == fa.FA_E_INVAL
    # too many rows for one diagonal block
    with pytest.raises(fa.FaError) as ei:
        p.ctx.encode_db_block(np.zeros((p.par.slots + 1, 16), np.float32), 16, 1, 4)
    assert ei.value.code == fa.FA_E_SHAPE
    # fold key missing for a projection
    with pytest.raises(fa.FaError) as ei:
        p.ctx.project_ct(ct, blk, 64, 16, 4)
    assert ei.value.code == fa.FA_E_NOKEY


def test_deterministic_repeat():
    """Two runs of the same scoring call give identical words (no races)."""
    p = pair("p1", wid=10)
    d, B = 128, 16
    X = gen.gaussian_unit_rows(gen.rng(10, gen.STREAM_DB), 4096, d)
    q = gen.gaussian_unit_rows(gen.rng(10, gen.STREAM_QUERY), 1, d)[0]
    ct_dev, _ = p.encrypt_both(ckks.encode(ckks.replicate(q, p.par.slots), p.n, 40), tag=10)
    p.keys(ckks.steps_for_bsgs(d, B), oracle=False)
    blk = p.ctx.encode_db_block(X.astype(np.float32), d, 1, B)
    a = p.export_ct(p.ctx.score_block(ct_dev, [blk, blk], d, 1, B), 2)
    b = p.export_ct(p.ctx.score_block(ct_dev, [blk, blk], d, 1, B), 2)
    assert np.array_equal(a, b)
    assert np.array_equal(a[0], a[1])


def test_more_blocks_than_one_launch_holds_and_a_zero_block():
    """35 blocks in one call (the multiply-accumulate launch addresses at most 32 blocks, so
    the library splits them): blocks 0, 31, 32 and 33 bit-exact against the oracle, every
    decrypted score within 1e-4; an all-zero block scores to the zero ciphertext exactly,
    on both sides; and no block, or a block of no rows, is an error."""
    from paper_2608_21131_amd import fa
    p = pair("tiny", wid=11)
    S, d, B = p.par.slots, 16, 4
    G = d // B
    g = gen.rng(11, gen.STREAM_DB)
    rows = [S if i % 3 == 0 else 1 + (37 * i) % S for i in range(34)]
    Xs = [gen.gaussian_unit_rows(g, r, d) for r in rows]
    q = gen.gaussian_unit_rows(gen.rng(11, gen.STREAM_QUERY), 1, d)[0]
    ct_dev, ct_orc = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=11)
    keys = p.keys(ckks.steps_for_bsgs(d, B))
    coeffs = [ckks.layout_b_coeffs(X, p.par, d, B) for X in Xs] + [np.zeros((d, p.n), dtype=np.int64)]
    blocks = [p.ctx.encode_db_block_int(c) for c in coeffs]
    say(f"[blocks] tiny d={d} B={B}: {len(blocks)} blocks in one call")
    out = p.ctx.score_block(ct_dev, blocks, d, 1, B)
    got = p.export_ct(out, len(blocks))
    qrot = p.orc.baby_rotations(ct_orc, B, keys)
    for i in (0, 31, 32, 33, 34):
        pts = np.stack([ckks.to_residues(ci, p.par.q) for ci in coeffs[i]]).reshape(G, B, p.par.L, p.n)
        assert np.array_equal(got[i], p.orc.bsgs_block(qrot, pts, B, G, keys)), i
    assert not got[34].any()
    W_ = p.ctx.ct_words
    for i, X in enumerate(Xs):
        z = p.ctx.decode(p.ctx.decrypt(out[i * W_:(i + 1) * W_]), 80)
        assert np.max(np.abs(z[:len(X)] - X @ q)) < 1e-4, i
    with pytest.raises(fa.FaError) as ei:
        p.ctx.score_block(ct_dev, [], d, 1, B)
    assert ei.value.code == fa.FA_E_SHAPE
    with pytest.raises(fa.FaError) as ei:
        p.ctx.encode_db_block(np.zeros((0, d), np.float32), d, 1, B)
    assert ei.value.code == fa.FA_E_SHAPE


def test_encode_projection_vs_oracle():
    """fa_encode_projection packs W's hybrid diagonals, pre-rotated, like the oracle (|dm| <= 1)."""
    p = pair("small", wid=11)
    d_in, R, B = 64, 16, 4
    W = gen.projection_matrix(gen.rng(11, gen.STREAM_W), d_in, R, var=1.0 / R).astype(np.float32)
    say("[encode_projection] small")
    pts = p.ctx.encode_projection(W, B)
    got = p.ctx.export(pts, R)
    pre = ckks.prerotate(ckks.projection_diagonals(W.astype(np.float64), p.par.slots), B)
    for j in range(R):
        ref = ckks.to_residues(ckks.encode(pre[j // B, j % B], p.n, 40), p.par.q)
        dif = got[j][0].astype(np.int64) - ref[0].astype(np.int64)
        q0 = np.int64(p.par.q[0])
        dif = np.where(dif > q0 // 2, dif - q0, np.where(dif < -(q0 // 2), dif + q0, dif))
        assert np.abs(dif).max() <= 1, j


@pytest.mark.parametrize("name,d,B", [("tiny", 16, 4), ("p1", 128, 16)])
def test_prepared_query_scores_identically(name, d, B):
    """fa_prepare_query + fa_score_prepared == fa_score_block, word for word, reused for two block sets."""
    p = pair(name, wid=14)
    S = p.par.slots
    X = gen.gaussian_unit_rows(gen.rng(14, gen.STREAM_DB, d), 2 * S, d)
    q = gen.gaussian_unit_rows(gen.rng(14, gen.STREAM_QUERY), 1, d)[0]
    ct, _ = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=14)
    p.keys(ckks.steps_for_bsgs(d, B), oracle=False)
    b0 = p.ctx.encode_db_block(X[:S].astype(np.float32), d, 1, B)
    b1 = p.ctx.encode_db_block(X[S:S + 1000].astype(np.float32), d, 1, B)
    say(f"[prepared] {name}")
    prep = p.ctx.prepare_query(ct, B)
    for blocks in ([b0, b1], [b1]):
        ref = p.export_ct(p.ctx.score_block(ct, blocks, d, 1, B), len(blocks))
        got = p.export_ct(p.ctx.score_prepared(ct, prep, blocks, d, B), len(blocks))
        assert np.array_equal(got, ref)


@pytest.mark.parametrize("name,d,B,nq,rows_list,oracle", [
    ("tiny", 16, 4, 5, [300, 512], True),   # groups of 4 + 1 queries per plaintext pass
    ("tiny", 16, 16, 3, [100], True),        # 2 + 1, G = 1 (no giant steps)
    ("tiny", 16, 4, 4, [64] * 33, True),     # 33 blocks: two plaintext passes of 4 queries
    ("tiny1", 16, 4, 4, [300], True),        # one digit, batched preparation
    ("p1", 128, 16, 2, [4096, 1000], False),
    ("p2", 128, 16, 4, [3000], False),
])
def test_batch_scores_match_oracle_and_single(name, d, B, nq, rows_list, oracle):
    """fa_score_batch: each query's blocks equal fa_score_prepared's word for word and, at the
    small size, the oracle's BSGS block; decrypted scores match float64 within 1e-4."""
    p = pair(name, wid=15)
    S = p.par.slots
    G = d // B
    g = gen.rng(15, gen.STREAM_DB, d, B)
    Xs = [gen.gaussian_unit_rows(g, r, d) for r in rows_list]
    Q = gen.gaussian_unit_rows(gen.rng(15, gen.STREAM_QUERY), nq, d)
    keys = p.keys(ckks.steps_for_bsgs(d, B), oracle=oracle)
    coeffs = [ckks.layout_b_coeffs(X, p.par, d, B) for X in Xs]
    blocks = [p.ctx.encode_db_block_int(c) for c in coeffs]
    cts = [p.encrypt_both(ckks.encode(ckks.replicate(Q[j], S), p.n, 40), tag=100 + j) for j in range(nq)]
    preps = [p.ctx.prepare_query(ct[0], B) for ct in cts]
    say(f"[batch] {name} d={d} B={B} nq={nq} blocks={rows_list}")
    outs = p.ctx.score_batch([ct[0] for ct in cts], preps, blocks, d, B)
    for j in range(nq):
        got = p.export_ct(outs[j], len(Xs))
        single = p.export_ct(p.ctx.score_prepared(cts[j][0], preps[j], blocks, d, B), len(Xs))
        assert np.array_equal(got, single), j
        if oracle:
            qrot = p.orc.baby_rotations(cts[j][1], B, keys)
            for i, c in enumerate(coeffs):
                pts = np.stack([ckks.to_residues(ci, p.par.q) for ci in c]).reshape(G, B, p.par.L, p.n)
                assert np.array_equal(got[i], p.orc.bsgs_block(qrot, pts, B, G, keys)), (j, i)
        for i, X in enumerate(Xs):
            W = p.ctx.ct_words
            z = p.ctx.decode(p.ctx.decrypt(outs[j][i * W:(i + 1) * W]), 80)
            assert np.max(np.abs(z[:len(X)] - X @ Q[j])) < 1e-4


@pytest.mark.parametrize("name,B,nq", [("tiny", 4, 1), ("tiny", 16, 3), ("tiny1", 16, 3), ("p1", 16, 5),
                                       ("p4", 16, 4)])
def test_prepare_batch_matches_single(name, B, nq):
    """fa_prepare_batch: every query's baby rotations equal fa_prepare_query's word for word
    (launch groups of 16 // nq steps x nq queries, the last group short), and the batch
    prepared at the small size scores to the oracle's BSGS block."""
    import torch
    p = pair(name, wid=17)
    S = p.par.slots
    d = 4 * B if name == "tiny" else 128
    keys = p.keys(ckks.steps_for_bsgs(d, B), oracle=(name == "tiny"))
    Q = gen.gaussian_unit_rows(gen.rng(17, gen.STREAM_QUERY, nq), nq, d)
    cts = [p.encrypt_both(ckks.encode(ckks.replicate(Q[j], S), p.n, 40), tag=170 + j) for j in range(nq)]
    say(f"[prepare_batch] {name} B={B} nq={nq}")
    preps = p.ctx.prepare_batch([ct[0] for ct in cts], B)
    torch.cuda.synchronize()
    words = (B - 1) * p.ctx.ct_words  # the B-1 rotated ciphertexts (the buffer holds one spare word)
    for j in range(nq):
        single = p.ctx.prepare_query(cts[j][0], B)
        assert torch.equal(preps[j].t[:words], single.t[:words]), j
    if name == "tiny":
        G = d // B
        X = gen.gaussian_unit_rows(gen.rng(17, gen.STREAM_DB), 200, d)
        c = ckks.layout_b_coeffs(X, p.par, d, B)
        blk = p.ctx.encode_db_block_int(c)
        pts = np.stack([ckks.to_residues(ci, p.par.q) for ci in c]).reshape(G, B, p.par.L, p.n)
        for j in range(nq):
            got = p.export_ct(p.ctx.score_prepared(cts[j][0], preps[j], [blk], d, B))[0]
            ref = p.orc.bsgs_block(p.orc.baby_rotations(cts[j][1], B, keys), pts, B, G, keys)
            assert np.array_equal(got, ref), j


def test_prepare_batch_rejects_bad_arguments():
    from paper_2608_21131_amd import fa
    p = pair("tiny", wid=18)
    S = p.par.slots
    q = gen.gaussian_unit_rows(gen.rng(18, gen.STREAM_QUERY), 1, 16)[0]
    ct, _ = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=18)
    p.keys([1, 2, 3], oracle=False)
    with pytest.raises(fa.FaError, match="FA_E_SHAPE"):
        p.ctx.prepare_batch([], 4)                                         # no query
    with pytest.raises(ValueError):
        p.ctx.prepare_batch([ct, ct], 4, outs=[p.ctx.prepare_query(ct, 4)])  # one buffer missing
    small = p.ctx.prepare_batch_workspace(2, 4)[:16]
    with pytest.raises(fa.FaError, match="FA_E_NOMEM"):
        p.ctx.prepare_batch([ct, ct], 4, ws=small)                         # workspace too small
    with pytest.raises(fa.FaError, match="FA_E_NOKEY"):
        p.ctx.prepare_batch([ct, ct], 8)                                   # no key for steps 4..7


def test_batch_rejects_bad_arguments():
    from paper_2608_21131_amd import fa
    p = pair("tiny", wid=16)
    S = p.par.slots
    d, B = 16, 4
    p.keys(ckks.steps_for_bsgs(d, B), oracle=False)
    q = gen.gaussian_unit_rows(gen.rng(16, gen.STREAM_QUERY), 1, d)[0]
    ct, _ = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=16)
    prep = p.ctx.prepare_query(ct, B)
    blk = p.ctx.encode_db_block(gen.gaussian_unit_rows(gen.rng(16, 0), 10, d).astype(np.float32), d, 1, B)
    with pytest.raises(ValueError):
        p.ctx.score_batch([ct, ct], [prep], [blk], d, B)       # one prepared set missing
    with pytest.raises(fa.FaError):
        p.ctx.score_batch([ct], [prep], [blk], d, 3)           # baby step does not divide d
    small = p.ctx.batch_workspace(1, 1, d, B)[:16]
    with pytest.raises(fa.FaError):
        p.ctx.score_batch([ct], [prep], [blk], d, B, ws=small)  # workspace too small


@pytest.mark.parametrize("name,d,B,rows_list", [
    ("tiny", 16, 4, [300, 512]),
    ("tiny", 16, 16, [100]),
    ("tiny", 16, 4, [32] * 33),  # 33 encrypted blocks: two ct x ct launches
    ("p1", 128, 16, [4096, 1000]),
    ("p2", 128, 16, [3000]),     # four key-switch digits in the relinearisation and giant steps
    ("s12", 64, 8, [700, 2048]),  # a short last digit
])
def test_encrypted_block_score_parity(name, d, B, rows_list):
    """Encrypted database blocks (ct x ct, lazy relinearisation): the encrypted diagonals, and
    every output ciphertext, equal the oracle's word for word; decrypted scores match float64."""
    from paper_2608_21131_amd import fa
    p = pair(name, wid=17)
    S = p.par.slots
    G = d // B
    g = gen.rng(17, gen.STREAM_DB, d, B)
    Xs = [gen.gaussian_unit_rows(g, r, d) for r in rows_list]
    q = gen.gaussian_unit_rows(gen.rng(17, gen.STREAM_QUERY), 1, d)[0]
    ct_dev, ct_orc = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=17)
    keys = p.keys(ckks.steps_for_bsgs(d, B))
    par = p.par
    ra = gen.uniform_residues(gen.rng(17, gen.STREAM_KEY_A, 0), par.primes, par.dnum, par.n)
    re = gen.rounded_gaussian(gen.rng(17, gen.STREAM_KEY_E, 0), (par.dnum, par.n))
    p.ctx.keygen_relin(p.s, ra, re)
    assert p.ctx.has_relin_key()
    rlk = p.orc.keygen_relin(p.s, ra, re)
    blocks, oblocks = [], []
    for bi, X in enumerate(Xs):
        c = ckks.layout_b_coeffs(X, par, d, B)
        a = np.stack([gen.uniform_residues(gen.rng(17, gen.STREAM_ENC_A, 1000 * bi + 1 + j), par.q, 1, p.n)[0]
                      for j in range(d)])
        e = np.stack([gen.rounded_gaussian(gen.rng(17, gen.STREAM_ENC_E, 1000 * bi + 1 + j), p.n) for j in range(d)])
        cts = p.ctx.encrypt_pts(p.ctx.encode_db_block_int(c), d, a, e)
        ocs = np.stack([p.orc.encrypt(c[j], a[j], e[j], p.s) for j in range(d)])
        assert np.array_equal(p.export_ct(cts, d), ocs)
        blocks.append(cts)
        oblocks.append(ocs.reshape(G, B, 2, par.L, p.n))
    say(f"[enc] {name} d={d} B={B} blocks={rows_list}")
    out = p.ctx.score_block(ct_dev, blocks, d, fa.LAYOUT_DIAG_ENC, B)
    got = p.export_ct(out, len(Xs))
    qrot = p.orc.baby_rotations(ct_orc, B, keys)
    for i, X in enumerate(Xs):
        assert np.array_equal(got[i], p.orc.bsgs_block_ct(qrot, oblocks[i], B, G, keys, rlk)), i
        W = p.ctx.ct_words
        z = p.ctx.decode(p.ctx.decrypt(out[i * W:(i + 1) * W]), 80)
        assert np.max(np.abs(z[:len(X)] - X @ q)) < 1e-4


def test_encrypted_block_needs_relin_key():
    from paper_2608_21131_amd import fa
    p = pair("tiny", wid=18)
    S = p.par.slots
    d, B = 16, 4
    p.keys(ckks.steps_for_bsgs(d, B), oracle=False)
    q = gen.gaussian_unit_rows(gen.rng(18, gen.STREAM_QUERY), 1, d)[0]
    ct, _ = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=18)
    c = ckks.layout_b_coeffs(gen.gaussian_unit_rows(gen.rng(18, 0), 10, d), p.par, d, B)
    a = np.zeros((d, p.par.L, p.n), dtype=np.uint64)
    e = np.zeros((d, p.n), dtype=np.int64)
    cts = p.ctx.encrypt_pts(p.ctx.encode_db_block_int(c), d, a, e)
    with pytest.raises(fa.FaError) as ei:
        p.ctx.score_block(ct, [cts], d, fa.LAYOUT_DIAG_ENC, B)
    assert ei.value.code == fa.FA_E_NOKEY


@pytest.mark.parametrize("name,d_in,R,B", [
    ("small", 64, 16, 4),
    ("small", 16, 16, 4),   # R = d_in: no fold
    ("small", 64, 16, 1),   # B = 1: no baby rotations
    ("p2", 512, 128, 16),
])
def test_encrypted_projection_parity(name, d_in, R, B):
    """fa_project_ct_enc (W's diagonals encrypted): the output ciphertext equals the oracle's
    ct x ct diagonal product and fold word for word and decrypts to W^T q."""
    from paper_2608_21131_amd import fa
    p = pair(name, wid=20)
    S, par = p.par.slots, p.par
    G, c = R // B, d_in // R
    W = gen.projection_matrix(gen.rng(20, gen.STREAM_W), d_in, R, var=1.0 / R)
    q = gen.gaussian_unit_rows(gen.rng(20, gen.STREAM_QUERY), 1, d_in)[0]
    ct_dev, ct_orc = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=20)
    fold = [R << k for k in range(int(np.log2(c)))]
    keys = p.keys(ckks.steps_for_bsgs(R, B) + fold)
    ra = gen.uniform_residues(gen.rng(20, gen.STREAM_KEY_A, 0), par.primes, par.dnum, par.n)
    re = gen.rounded_gaussian(gen.rng(20, gen.STREAM_KEY_E, 0), (par.dnum, par.n))
    p.ctx.keygen_relin(p.s, ra, re)
    rlk = p.orc.keygen_relin(p.s, ra, re)
    pre = ckks.prerotate(ckks.projection_diagonals(W, S), B)
    wco = np.stack([ckks.encode(pre[g, b], p.n, 40) for g in range(G) for b in range(B)])
    a = np.stack([gen.uniform_residues(gen.rng(20, gen.STREAM_ENC_A, 1 + j), par.q, 1, p.n)[0] for j in range(R)])
    e = np.stack([gen.rounded_gaussian(gen.rng(20, gen.STREAM_ENC_E, 1 + j), p.n) for j in range(R)])
    wct = p.ctx.encrypt_pts(p.ctx.encode_db_block_int(wco), R, a, e)
    owct = np.stack([p.orc.encrypt(wco[j], a[j], e[j], p.s) for j in range(R)])
    assert np.array_equal(p.export_ct(wct, R), owct)
    say(f"[proj-enc] {name} d_in={d_in} R={R} B={B}")
    qr = p.ctx.project_ct_enc(ct_dev, wct, d_in, R, B)
    got = p.export_ct(qr)[0]
    z = p.orc.bsgs_block_ct(p.orc.baby_rotations(ct_orc, B, keys), owct.reshape(G, B, 2, par.L, p.n), B, G,
                            keys, rlk)
    z = p.orc.rotate_sum(z, R, len(fold), keys)
    assert np.array_equal(got, z)
    zz = p.ctx.decode(p.ctx.decrypt(qr), 80)
    assert np.max(np.abs(zz - np.tile(W.T @ q, S // R))) < 1e-4


def test_encrypted_projection_rejects_bad_arguments():
    from paper_2608_21131_amd import fa
    p = pair("small", wid=21)
    S, d_in, R, B = p.par.slots, 64, 16, 4
    p.keys(ckks.steps_for_bsgs(R, B) + [16, 32], oracle=False)
    q = gen.gaussian_unit_rows(gen.rng(21, gen.STREAM_QUERY), 1, d_in)[0]
    ct, _ = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=21)
    a = np.zeros((R, p.par.L, p.n), dtype=np.uint64)
    e = np.zeros((R, p.n), dtype=np.int64)
    wco = np.zeros((R, p.n), dtype=np.int64)
    wct = p.ctx.encrypt_pts(p.ctx.encode_db_block_int(wco), R, a, e)
    with pytest.raises(fa.FaError) as ei:                       # no relinearisation key yet
        p.ctx.project_ct_enc(ct, wct, d_in, R, B)
    assert ei.value.code == fa.FA_E_NOKEY
    with pytest.raises(fa.FaError) as ei:                       # r does not divide d_in
        p.ctx.project_ct_enc(ct, wct, 48, R, B, ws=p.ctx.workspace(fa.OP_PROJECT_ENC, 1, R, B))
    assert ei.value.code == fa.FA_E_SHAPE
    with pytest.raises(fa.FaError) as ei:                       # workspace of the plaintext projection
        p.ctx.project_ct_enc(ct, wct, d_in, R, B, ws=p.ctx.workspace(fa.OP_PROJECT, 1, R, B)[:1024])
    assert ei.value.code == fa.FA_E_NOMEM


# ----------------------------------------------------------------------------
# membership path: rescale, ct x ct product, Chebyshev evaluator, sign iteration
# ----------------------------------------------------------------------------
def _gpu_chain(logn, L, K, wid):
    from paper_2608_21131_amd import fa
    top = ckks.Params(logn=logn, L=L, K=K, log_scale=50)
    s = gen.ternary_secret(gen.rng(wid, gen.STREAM_SECRET), top.n)
    ra = gen.uniform_residues(gen.rng(wid, gen.STREAM_KEY_A, 0), top.primes, top.dnum, top.n)
    re_ = gen.rounded_gaussian(gen.rng(wid, gen.STREAM_KEY_E, 0), (top.dnum, top.n))
    ctx = fa.Context(logn, L, K, 50)
    assert ctx.primes == top.primes
    ctx.keygen_relin(s, ra, re_)
    levels = [ctx] + [ctx.at_level(l) for l in range(L - 1, 1, -1)]
    och = ckks.LevelChain(top, s, (ra, re_), {}, rot_levels=[])
    return top, s, levels, och


def _enc_both(top, levels, och, s, v, wid, tag):
    m = ckks.encode(v, top.n, 50)
    a = gen.uniform_residues(gen.rng(wid, gen.STREAM_ENC_A, tag), top.q, 1, top.n)[0]
    e = gen.rounded_gaussian(gen.rng(wid, gen.STREAM_ENC_E, tag), top.n)
    return levels[0].encrypt(m, a, e), och.orc[top.L].encrypt(m, a, e, s)


def _at(levels, ct, L, offset_words=0):
    """The ciphertext at level L held in the first words of ct (from offset_words), described
    at that level."""
    c = levels[levels[0].L - L]
    t = ct.t if hasattr(ct, "t") else ct
    return c.wrap(t[offset_words:offset_words + 2 * L * c.n], 2, 1, 0)


def _export_at(levels, ct, L):
    c = levels[levels[0].L - L]
    return c.export(_at(levels, ct, L)).reshape(2, L, c.n)


def test_rescale_and_product_parity():
    top, s, levels, och = _gpu_chain(11, 6, 2, 50)
    v1 = gen.gaussian_unit_rows(gen.rng(50, gen.STREAM_QUERY), 1, top.slots)[0]
    v2 = gen.gaussian_unit_rows(gen.rng(50, gen.STREAM_DB), 1, top.slots)[0]
    x, xo = _enc_both(top, levels, och, s, v1, 50, 1)
    y, yo = _enc_both(top, levels, och, s, v2, 50, 2)
    say("[chain] rescale / product")
    r = levels[0].rescale(levels[1], x)
    assert np.array_equal(_export_at(levels, r, top.L - 1), och.orc[top.L].rescale(xo))
    p = levels[0].mul_ct(x, y)
    po = och.orc[top.L].mul(xo, yo, och.rlk[top.L])
    assert np.array_equal(_export_at(levels, p, top.L), po)
    pr = levels[0].rescale(levels[1], p)
    z = levels[1].decode(levels[1].decrypt(_at(levels, pr, top.L - 1)), 50) * (2.0 ** 50 / (2.0 ** 100 / top.q[-1]))
    assert np.max(np.abs(z - v1 * v2)) < 1e-6
    # constants and sums
    a = levels[0].ct_add_const(levels[0].ct_mul_const(x, -3), 12345)
    ao = och.orc[top.L].add_const(och.orc[top.L].mul_const(xo, -3), 12345)
    assert np.array_equal(_export_at(levels, a, top.L), ao)
    d = levels[0].ct_add(x, y, subtract=True)
    assert np.array_equal(_export_at(levels, d, top.L), och.orc[top.L].add(xo, yo, sub=True))


def test_chebyshev_and_sign_parity():
    """The GPU chain evaluates the degree-7 Chebyshev series and two sign steps exactly as
    the oracle chain does (word for word), and the values match numpy."""
    from paper_2608_21131_amd import fa
    top, s, levels, och = _gpu_chain(11, 9, 2, 51)
    u = np.random.default_rng(51).uniform(-1, 1, top.slots)
    coeffs = np.random.default_rng(52).uniform(-1, 1, 8)
    x, xo = _enc_both(top, levels, och, s, u, 51, 1)
    say("[chain] Chebyshev degree 7")
    out, L, sc = fa.cheb_eval(levels, x, top.L, 2.0 ** 50, coeffs)
    oo, Lo, so = ckks.cheb_eval(och, xo, top.L, 2.0 ** 50, coeffs)
    assert (L, sc) == (Lo, so)
    assert np.array_equal(_export_at(levels, out, L), oo)
    c = levels[top.L - L]
    z = c.decode(c.decrypt(_at(levels, out, L)), 50) * (2.0 ** 50 / sc)
    assert np.max(np.abs(z - np.polynomial.chebyshev.chebval(u, coeffs))) < 1e-6
    say("[chain] two sign steps")
    v = np.random.default_rng(53).uniform(-0.5, 0.5, top.slots)
    w, wo = _enc_both(top, levels, och, s, 4 * v, 51, 2)
    out, L, sc, m = fa.sign_iter(levels, w, top.L, 2.0 ** 50, 4, 2)
    oo, Lo, so, mo = ckks.sign_iter(och, wo, top.L, 2.0 ** 50, 4, 2)
    assert (L, sc, m) == (Lo, so, mo)
    assert np.array_equal(_export_at(levels, out, L), oo)
    c = levels[top.L - L]
    z = c.decode(c.decrypt(_at(levels, out, L)), 50) * (2.0 ** 50 / sc) / m
    f = lambda t: (3 * t - t ** 3) / 2
    assert np.max(np.abs(z - f(f(v)))) < 1e-6


def _gpu_membership_chain(logn, L, K, wid, d, B):
    from paper_2608_21131_amd import fa
    top = ckks.Params(logn=logn, L=L, K=K, log_scale=50)
    s = gen.ternary_secret(gen.rng(wid, gen.STREAM_SECRET), top.n)
    ra = gen.uniform_residues(gen.rng(wid, gen.STREAM_KEY_A, 0), top.primes, top.dnum, top.n)
    re_ = gen.rounded_gaussian(gen.rng(wid, gen.STREAM_KEY_E, 0), (top.dnum, top.n))
    steps = sorted(set(ckks.steps_for_bsgs(d, B) + [1 << k for k in range(int(np.log2(d)))]))
    rot = {r: (gen.uniform_residues(gen.rng(wid, gen.STREAM_KEY_A, r), top.primes, top.dnum, top.n),
               gen.rounded_gaussian(gen.rng(wid, gen.STREAM_KEY_E, r), (top.dnum, top.n))) for r in steps}
    ctx = fa.Context(logn, L, K, 50)
    assert ctx.primes == top.primes
    ctx.keygen_relin(s, ra, re_)
    ctx.keygen(s, steps, np.stack([rot[r][0] for r in steps]), np.stack([rot[r][1] for r in steps]))
    levels = [ctx] + [ctx.at_level(l) for l in range(L - 1, 1, -1)]
    och = ckks.LevelChain(top, s, (ra, re_), rot, rot_levels=[L, L - 1])
    return top, s, levels, och


@pytest.mark.parametrize("y_lo,y_hi,degree,iters,nblk", [(0.5, 2.5, 7, 2, 2), (0.6, 1.6, 7, 2, 2),
                                                       (0.5, 2.5, 1, 1, 1), (0.5, 2.5, 3, 2, 1)])
def test_membership_scan_parity(y_lo, y_hi, degree, iters, nblk):
    """The membership scan (scores, |q_R|^2 by square and fold, Chebyshev tau |q_R|, sign
    steps; from level 11 at N = 2^11, d = 16, a full and a ragged block) writes the oracle's
    ciphertexts word for word, and its decrypted signs are the decisions cos(q_R, x_i) >= tau
    wherever the margin exceeds the series' error.  Also the degenerate settings: a series
    of degree 1, one sign step, one block."""
    from paper_2608_21131_amd import fa
    d, B, tau, m = 16, 4, 0.6, 4
    top, s, levels, och = _gpu_membership_chain(11, 11, 3, 46, d, B)
    g = np.random.default_rng(46)
    X = gen.normalize_rows(g.standard_normal((top.slots + 500, d)))
    qR = 1.1 * gen.normalize_rows((X[3] + 0.4 * g.standard_normal(d))[None])[0]
    coeffs = fa.cheb_fit_sqrt(tau, y_lo, y_hi, degree)
    x, xo = _enc_both(top, levels, och, s, ckks.replicate(qR, top.slots), 46, 1)
    parts = [X[:top.slots], X[top.slots:]][:nblk]
    X = np.vstack(parts)
    blocks = [levels[0].encode_db_block_int(ckks.layout_b_coeffs(b, top, d, B)) for b in parts]
    oblocks = [ckks.layout_b_pts(b, top, d, B) for b in parts]
    say(f"[membership] N=2^11 L=11 d={d} domain [{y_lo}, {y_hi}] degree {degree}, {iters} sign steps, "
        f"{nblk} block(s)")
    out, L, sc, mo = fa.membership(levels, x, top.L, 2.0 ** 50, blocks, d, B, y_lo, y_hi, coeffs, m, iters)
    oo, Lo, so, mo2 = ckks.membership(och, xo, top.L, 2.0 ** 50, oblocks, d, B, y_lo, y_hi, coeffs, m, iters)
    depth = 1 + (int(np.ceil(np.log2(degree))) + 1) + 2 * iters
    assert (L, sc, mo) == (Lo, so, mo2) and L == top.L - depth
    ctw = levels[0].ct_words
    c = levels[top.L - L]
    z = []
    for i in range(nblk):
        blk = _at(levels, out, L, i * ctw)
        assert np.array_equal(_export_at(levels, blk, L), oo[i]), i
        z.append(c.decode(c.decrypt(blk), 50) * (2.0 ** 50 / sc) / mo)
    z = np.concatenate(z)[:len(X)]
    y = float(qR @ qR)
    t = np.polynomial.chebyshev.chebval((2 * y - y_lo - y_hi) / (y_hi - y_lo), coeffs)
    margin = X @ qR - tau * np.sqrt(y)
    ok = np.abs(margin) > abs(t - tau * np.sqrt(y)) + 2e-4
    assert np.all(np.sign(z[ok]) == np.sign(margin[ok]))
    assert 0 < np.count_nonzero(margin > 0) < len(X) // 4


def test_chain_calls_reject_short_chains_and_bad_arguments():
    """The chain calls check depth, multipliers and keys before any launch: a degree-7
    series needs 4 levels below its input, two sign steps 4, and a multiplier that would
    overflow is refused; the membership scan needs its fold keys."""
    from paper_2608_21131_amd import fa
    top, s, levels, och = _gpu_chain(10, 5, 2, 52)
    x, _ = _enc_both(top, levels, och, s, np.full(top.slots, 0.5), 52, 1)
    with pytest.raises(fa.FaError) as ei:
        fa.cheb_eval(levels, x, top.L, 2.0 ** 50, np.ones(8))
    assert ei.value.code == fa.FA_E_SHAPE
    fa.cheb_eval(levels, x, top.L, 2.0 ** 50, np.ones(4))  # degree 3: 3 levels, 5 -> 2
    with pytest.raises(fa.FaError) as ei:
        fa.sign_iter(levels, x, top.L, 2.0 ** 50, 4, 3)
    assert ei.value.code in (fa.FA_E_SHAPE, fa.FA_E_INVAL)
    with pytest.raises(fa.FaError) as ei:
        fa.sign_iter(levels, x, top.L, 2.0 ** 50, 1 << 21, 1)
    assert ei.value.code == fa.FA_E_INVAL
    blk = levels[0].new_pt(16)
    with pytest.raises(fa.FaError) as ei:
        fa.membership(levels, x, top.L, 2.0 ** 50, [blk], 16, 4, 0.5, 2.5, np.ones(2), 4, 1)
    assert ei.value.code == fa.FA_E_NOKEY


# ----------------------------------------------------------------------------
# the buffer descriptors, block ids and explicit primes of the C ABI
# ----------------------------------------------------------------------------
def test_descriptor_checks_refuse_mismatched_buffers():
    """Every scoring-path call checks its fa_buf descriptors on the host before any launch: a
    ciphertext at another level, a plaintext passed as a ciphertext, blocks at two scales, a
    block with too few diagonals, a product scale the modulus cannot hold, an output too small,
    a block id out of range and an in-place rotation are refused with FA_E_SHAPE / FA_E_INVAL,
    and the output buffers are left untouched."""
    import torch
    from paper_2608_21131_amd import fa
    p = pair("tiny", wid=30)
    S, d, B = p.par.slots, 16, 4
    p.keys(ckks.steps_for_bsgs(d, B) + [16, 32], oracle=False)
    q = gen.gaussian_unit_rows(gen.rng(30, gen.STREAM_QUERY), 1, d)[0]
    ct, _ = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=30)
    X = gen.gaussian_unit_rows(gen.rng(30, gen.STREAM_DB), 100, d).astype(np.float32)
    blk = p.ctx.encode_db_block(X, d, fa.LAYOUT_DIAG, B)
    assert (blk.n_polys, blk.count, blk.limbs, blk.log_scale) == (1, d, p.par.L, 40)
    low = p.ctx.at_level(2)
    ct_low = p.ctx.drop_level(low, ct)
    assert (ct_low.limbs, ct_low.log_scale) == (2, 40)
    out = p.ctx.new_ct(2)
    out.t.fill_(7.0)

    def code(fn, *a, **k):
        with pytest.raises(fa.FaError) as ei:
            fn(*a, **k)
        return ei.value.code

    say("[descriptors] tiny")
    # a ciphertext of the 2-prime level given to the 3-prime context (same tensor, its descriptor)
    wrong_level = p.ctx.wrap(ct_low.t, fa.CT, 1, 40)
    wrong_level.limbs = 2
    assert code(p.ctx.score_block, wrong_level, [blk], d, fa.LAYOUT_DIAG, B, out=out) == fa.FA_E_SHAPE
    assert code(p.ctx.rotate_sum, wrong_level, 1, 1, 1) == fa.FA_E_SHAPE
    assert code(p.ctx.project_ct, wrong_level, blk, 64, d, B) == fa.FA_E_SHAPE
    # a plaintext passed as the query, a ciphertext passed as a block
    assert code(p.ctx.score_block, blk.item(0), [blk], d, fa.LAYOUT_DIAG, B, out=out) == fa.FA_E_SHAPE
    assert code(p.ctx.score_block, ct, [ct], d, fa.LAYOUT_DIAG, B, out=out) == fa.FA_E_SHAPE
    assert code(p.ctx.rotate_sum, blk, 1, 1, 1) == fa.FA_E_SHAPE
    assert code(p.ctx.decrypt, blk.item(0)) == fa.FA_E_SHAPE
    # W's plaintexts at another level, or too few of them
    w_low = low.encode_db_block(X, d, fa.LAYOUT_DIAG, B)
    assert code(p.ctx.project_ct, ct, w_low, 64, d, B) == fa.FA_E_SHAPE
    assert code(p.ctx.project_ct, ct, blk.items(0, d - 1), 64, d, B) == fa.FA_E_SHAPE
    # blocks at two scales; a block with fewer than d diagonals
    blk80 = p.ctx.encode_db_block_int(np.zeros((d, p.n), np.int64), log_scale=80)
    assert code(p.ctx.score_block, ct, [blk, blk80], d, fa.LAYOUT_DIAG, B, out=out) == fa.FA_E_SHAPE
    assert code(p.ctx.score_block, ct, [blk.items(0, d - 1)], d, fa.LAYOUT_DIAG, B, out=out) == fa.FA_E_SHAPE
    # a product scale above Q / 2^8 (Q ~ 2^150 here): 2^(110 + 40)
    hi = p.ctx.wrap(ct.t, fa.CT, 1, 110)
    assert code(p.ctx.score_block, hi, [blk], d, fa.LAYOUT_DIAG, B, out=out) == fa.FA_E_SHAPE
    assert code(p.ctx.project_ct, hi, blk, 64, d, B) == fa.FA_E_SHAPE
    # an output too small for two blocks; block ids out of range
    assert code(p.ctx.score_block, ct, [blk, blk], d, fa.LAYOUT_DIAG, B, out=out.item(0)) == fa.FA_E_SHAPE
    assert code(p.ctx.score_block, ct, [blk], d, fa.LAYOUT_DIAG, B, out=out, block_ids=[1]) == fa.FA_E_INVAL
    assert code(p.ctx.score_block, ct, [blk], d, fa.LAYOUT_DIAG, B, out=out, block_ids=[-1]) == fa.FA_E_INVAL
    # a rotation into its own input
    assert code(p.ctx.rotate, ct, 1, out=ct) == fa.FA_E_INVAL
    torch.cuda.synchronize()
    assert bool((out.t == 7.0).all()), "a refused call wrote its output"


def test_block_ids_select_resident_blocks():
    """block_ids: the scorer takes the ids of the groups to score among the resident blocks
    (repeats allowed) and writes output j for block ids[j], word for word what scoring that
    list of blocks directly gives; the oracle agrees on one of them."""
    p = pair("tiny", wid=31)
    S, d, B = p.par.slots, 16, 4
    G = d // B
    keys = p.keys(ckks.steps_for_bsgs(d, B))
    q = gen.gaussian_unit_rows(gen.rng(31, gen.STREAM_QUERY), 1, d)[0]
    ct, ct_o = p.encrypt_both(ckks.encode(ckks.replicate(q, S), p.n, 40), tag=31)
    g = gen.rng(31, gen.STREAM_DB)
    Xs = [gen.gaussian_unit_rows(g, r, d) for r in (300, 512, 77)]
    coeffs = [ckks.layout_b_coeffs(X, p.par, d, B) for X in Xs]
    resident = [p.ctx.encode_db_block_int(c) for c in coeffs]
    ids = [2, 0, 2, 1]
    say("[block_ids] tiny")
    got = p.export_ct(p.ctx.score_block(ct, resident, d, 1, B, block_ids=ids), len(ids))
    ref = p.export_ct(p.ctx.score_block(ct, [resident[i] for i in ids], d, 1, B), len(ids))
    assert np.array_equal(got, ref)
    pts = np.stack([ckks.to_residues(ci, p.par.q) for ci in coeffs[2]]).reshape(G, B, p.par.L, p.n)
    assert np.array_equal(got[0], p.orc.bsgs_block(p.orc.baby_rotations(ct_o, B, keys), pts, B, G, keys))
    prep = p.ctx.prepare_query(ct, B)
    got2 = p.export_ct(p.ctx.score_prepared(ct, prep, resident, d, B, block_ids=ids), len(ids))
    assert np.array_equal(got2, ref)
    got3 = p.ctx.score_batch([ct, ct], [prep, prep], resident, d, B, block_ids=ids)
    assert all(np.array_equal(p.export_ct(o, len(ids)), ref) for o in got3)


def test_explicit_primes_match_the_oracle():
    """fa_params.primes: a context over an explicit prime list (not the default choice: every
    other NTT prime below 2^50, ciphertext and special primes interleaved) rotates and scores
    exactly as the oracle over the same primes."""
    from paper_2608_21131_amd import fa
    logn, L, K = 10, 3, 1
    primes = ckks.find_primes(logn, 2 * (L + K))[1::2]
    par = ckks.Params(logn=logn, L=L, K=K, primes=primes)
    orc = ckks.Oracle(par)
    ctx = fa.Context(logn, L, K, 40, primes=primes)
    assert ctx.primes == primes
    s = gen.ternary_secret(gen.rng(32, gen.STREAM_SECRET), par.n)
    d, B = 16, 4
    steps = ckks.steps_for_bsgs(d, B)
    rand = [(gen.uniform_residues(gen.rng(32, gen.STREAM_KEY_A, r), par.primes, par.dnum, par.n),
             gen.rounded_gaussian(gen.rng(32, gen.STREAM_KEY_E, r), (par.dnum, par.n))) for r in steps]
    ctx.keygen(s, steps, np.stack([x[0] for x in rand]), np.stack([x[1] for x in rand]))
    keys = {r: orc.keygen(s, r, *rand[i]) for i, r in enumerate(steps)}
    q = gen.gaussian_unit_rows(gen.rng(32, gen.STREAM_QUERY), 1, d)[0]
    m = ckks.encode(ckks.replicate(q, par.slots), par.n, 40)
    a = gen.uniform_residues(gen.rng(32, gen.STREAM_ENC_A), par.q, 1, par.n)[0]
    e = gen.rounded_gaussian(gen.rng(32, gen.STREAM_ENC_E), par.n)
    ct, ct_o = ctx.encrypt(m, a, e), orc.encrypt(m, a, e, s)
    say("[primes] explicit list, N=2^10")
    assert np.array_equal(ctx.export(ctx.rotate(ct, 3)).reshape(2, L, par.n), orc.rotate(ct_o, 3, keys[3]))
    X = gen.gaussian_unit_rows(gen.rng(32, gen.STREAM_DB), 400, d)
    c = ckks.layout_b_coeffs(X, par, d, B)
    out = ctx.score_block(ct, [ctx.encode_db_block_int(c)], d, fa.LAYOUT_DIAG, B)
    pts = np.stack([ckks.to_residues(ci, par.q) for ci in c]).reshape(d // B, B, L, par.n)
    ref = orc.bsgs_block(orc.baby_rotations(ct_o, B, keys), pts, B, d // B, keys)
    assert np.array_equal(ctx.export(out).reshape(2, L, par.n), ref)
    z = ctx.decode(ctx.decrypt(out), 80)
    assert np.max(np.abs(z[:400] - X @ q)) < 1e-4


@pytest.mark.parametrize("nq", [17, 33])
def test_prepare_batch_beyond_one_group(nq):
    """fa_prepare_batch with more queries than one key-switch group holds (groups of 16):
    every query's baby rotations equal fa_prepare_query's word for word."""
    import torch
    p = pair("tiny", wid=33)
    S, B = p.par.slots, 4
    p.keys(ckks.steps_for_bsgs(16, B), oracle=False)
    Q = gen.gaussian_unit_rows(gen.rng(33, gen.STREAM_QUERY, nq), nq, 16)
    cts = [p.encrypt_both(ckks.encode(ckks.replicate(Q[j], S), p.n, 40), tag=330 + j)[0] for j in range(nq)]
    say(f"[prepare_batch] tiny B={B} nq={nq}")
    preps = p.ctx.prepare_batch(cts, B)
    torch.cuda.synchronize()
    words = (B - 1) * p.ctx.ct_words  # the rotations (the buffer holds one spare word)
    for j in range(nq):
        assert torch.equal(preps[j].t[:words], p.ctx.prepare_query(cts[j], B).t[:words]), j
