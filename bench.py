"""Benchmark: encrypted candidate scoring on one MI355X.

Default workload (``--workload rerank``): the rerank level of the three-level
search -- one slot-packed CKKS query ciphertext scored against 110,000
candidate rows of dimension 512 (4 diagonal blocks of up to 32,768 rows,
2,048 plaintexts), ring N = 2^16, 12 ciphertext primes + 3 special primes of
50 bits, scale 2^40.  A step is one whole level: hoisted baby rotations of the
query, the multiply-accumulate stream over every resident plaintext, the
giant-step rotations and ModDown, ending with the block output ciphertexts in
HBM.  Other workloads: tiny (row layout + rotate-and-sum), fine (65,536 x 96-d
at N=2^15), rank (encrypted 512->128 projection, then 16,384 candidates) and
three_level (32 queries through coarse, fine and rerank levels with the
client's decrypt and top-k between levels).

Prints one JSON line.  Inputs are synthetic (seeded), see
paper_2608_21131_amd/workloads.py.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# fp64 vector rate of the MI355X: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = 39.3e12 lane-operations
# per second (78.6 TFLOP/s counting an FMA as two).  A modular product of two residues in this
# library's exact fp64 arithmetic is 6 of them (product, its FMA error term, quotient estimate,
# rounding, FMA correction, sum), so the ALU roofline of the key-switch phases is 6.55e12 products/s.
FP64_LANE_OPS = 256 * 4 * 16 * 2.4e9
MODMUL_PEAK = FP64_LANE_OPS / 6
METRIC = "encrypted candidate scores/sec + ms/level at 110k x 512-dim, one MI355X"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="rerank",
                    help="face: the membership scan alone (its own JSON line)",
                    choices=["tiny", "fine", "rank", "rerank", "three_level", "face"])
    ap.add_argument("--baby-step", type=int, default=0)
    ap.add_argument("--level", type=int, default=0,
                    help="fine/rerank/three_level: drop the query to this many ciphertext primes and score there, "
                         "with the database enrolled at that level (0: score at all primes)")
    ap.add_argument("--queries", type=int, default=0, help="three_level: queries per step (default 32)")
    ap.add_argument("--also-level", type=int, default=3,
                    help="rerank: also time the level with the query dropped to this many primes and report it "
                         "under level_drop (0: skip)")
    ap.add_argument("--batch", type=int, default=4,
                    help="rerank: also time cross-query batching (this many queries per plaintext pass, each "
                         "prepared once, all scored against the same blocks) and report it under query_batch "
                         "(0: skip); three_level: queries per coarse-level pass (at most 4)")
    ap.add_argument("--enc-level", type=int, default=3,
                    help="rerank: also time the encrypted-database variant (ct x ct, database diagonals encrypted "
                         "and enrolled at this many primes, lazy relinearisation) and report it under enc_db "
                         "(0: skip; 12: all primes)")
    ap.add_argument("--enc-w", type=int, default=1,
                    help="rank: also time the projection with W's diagonals encrypted and report it under "
                         "enc_projection (0: skip)")
    ap.add_argument("--three-level", type=int, default=1,
                    help="rerank: also run the full three-level query (32 queries back to back at all 12 primes, "
                         "coarse, fine and rerank levels with the client's decrypt and top-k between them) and "
                         "report it under three_level (0: skip)")
    ap.add_argument("--membership", type=int, default=1,
                    help="rerank: also time the face membership scan (222,049 centroids, encrypted threshold) "
                         "and report it under membership (0: skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-check", action="store_true", help="skip the decrypt-and-compare check")
    ap.add_argument("--copy-calib", action="store_true",
                    help="before the timed region, fill, copy and sum one plain 1 GiB buffer (HBM counter "
                         "calibration: known writes, reads and writes, reads)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "k_mac_diag3_rerank110k_traffic.md"),
                    help="rocprofv3 counter summary with the measured per-launch HBM bytes of the "
                         "multiply-accumulate kernel (used only while that kernel's source is unchanged)")
    return ap.parse_args()


class Bench:
    def __init__(self, args):
        import torch
        from paper_2608_21131_amd import fa, workloads as wl
        self.torch, self.fa, self.wl = torch, fa, wl
        self.args = args
        w = wl.WORKLOADS[args.workload]
        if args.baby_step:
            w.B = args.baby_step
        self.w = w
        torch.cuda.set_device(0)
        t0 = time.time()
        self.t0 = t0
        if w.name == "face":  # run_membership builds its own chain of contexts
            return
        self.ctx = fa.Context(w.log_n, w.L, w.K, 40)
        self.s = wl.secret(w)
        steps = wl.rotation_steps(w)
        for i in range(0, len(steps), 8):
            chunk = steps[i:i + 8]
            rand = [wl.key_randomness(w, r, self.ctx.primes, self.ctx.dnum) for r in chunk]
            self.ctx.keygen(self.s, chunk, np.stack([x[0] for x in rand]), np.stack([x[1] for x in rand]))
        ra, re_ = wl.relin_randomness(w, self.ctx.primes, self.ctx.dnum)
        self.ctx.keygen_relin(self.s, ra, re_)
        log(f"[bench] {w.name}: keys for {len(steps)} rotations + relinearisation ({time.time() - t0:.1f}s)")
        self.t0 = t0

    def encrypt(self, v, tag=0):
        w = self.w
        a, e = self.wl.enc_randomness(w, self.ctx.primes[:w.L], tag)
        return self.ctx.encrypt(self.ctx.encode(np.tile(v, w.slots // len(v)), 40), a, e)

    def decode(self, ct, i, log_scale):
        W = self.ctx.ct_words
        return self.ctx.decode(self.ctx.decrypt(ct[i * W:(i + 1) * W]), log_scale)

    def timed(self, step_fn, steps, warmup):
        torch = self.torch
        for _ in range(warmup):
            step_fn()
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for _ in range(steps):
            step_fn()
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / steps

    def phases(self, step_fn, ctx, n=3):
        """The library's phase split (baby / MAC / giant), from n further steps each followed by its
        (synchronising) read.  The timed steps run back to back without it: a read after every step
        would hold the host until the GPU drains, and the next step's first launches would start late."""
        ctx.profile(True)
        out = []
        for _ in range(n):
            step_fn()
            out.append(ctx.profile_read())
        ctx.profile(False)
        return {k: float(np.mean([p[k] for p in out])) for k in out[0]}


def pad(v, d):
    out = np.zeros(d)
    out[:len(v)] = v
    return out


def run_diag_level(bn, args):
    """fine / rerank: one diagonal-layout level over all blocks (optionally after a level drop)."""
    w, fa = bn.w, bn.fa
    top = bn.ctx
    ctx = top.at_level(args.level) if args.level and args.level < w.L else top
    X, centers = bn.wl.candidate_rows(w)
    S = w.slots
    blocks = [ctx.encode_db_block(X[b * S:(b + 1) * S], w.d, fa.LAYOUT_DIAG, w.B) for b in range(w.n_blocks)]
    bn.torch.cuda.synchronize()
    log(f"[bench] encoded {w.n_blocks} blocks, {w.n_blocks * w.d} plaintexts ({time.time() - bn.t0:.1f}s)")
    qv = bn.wl.query_vectors(w, 1, centers)[0]
    q_top = bn.encrypt(pad(qv, w.d))
    q = ctx.new_ct() if ctx is not top else q_top
    out = ctx.new_ct(w.n_blocks)
    ws = ctx.workspace(fa.OP_SCORE, w.n_blocks, w.d, w.B)
    if args.copy_calib:
        src = bn.torch.empty(1 << 27, dtype=bn.torch.float64, device="cuda")
        dst = bn.torch.empty_like(src)
        src.fill_(1.0)  # 1 GiB written
        dst.copy_(src)  # 1 GiB read, 1 GiB written
        tot = src.sum()  # 1 GiB read, nothing but the scalar written
        bn.torch.cuda.synchronize()
        del src, dst, tot

    def step():
        if ctx is not top:
            top.drop_level(ctx, q_top, out=q)
        ctx.score_block(q, blocks, w.d, fa.LAYOUT_DIAG, w.B, out=out, ws=ws)

    ms = bn.timed(step, args.steps, args.warmup)
    ph = bn.phases(step, ctx)
    err = None
    if not args.no_check:
        err = 0.0
        W_ = ctx.ct_words
        for b in range(w.n_blocks):
            rows = X[b * S:(b + 1) * S].astype(np.float64)
            z = ctx.decode(ctx.decrypt(out[b * W_:(b + 1) * W_]), 80)
            err = max(err, float(np.max(np.abs(z[:len(rows)] - rows @ qv))))
    ptw = ctx.L * w.n
    mac_bytes = 8 * (w.n_blocks * w.d * ptw + (w.B - 1) * 2 * ptw + 2 * ptw + w.n_blocks * w.G * 2 * ptw)
    stream_bytes = 8 * w.n_blocks * w.d * ptw
    return dict(ms=ms, scores=w.rows, phases=ph, err=err, mac_bytes=mac_bytes, stream_bytes=stream_bytes,
                X=X, cpu=(lambda: cpu_level_diag(bn, X, qv, L=ctx.L)), ctx=ctx, blocks=blocks, centers=centers,
                io=transfer_ms(bn, q, out))


def transfer_ms(bn, q, out):
    """Outside the timed level: the PCIe legs a client adds around it, timed with events on
    the stream: the query ciphertext host -> device and the output ciphertexts device -> host,
    both from / to pinned host memory."""
    torch = bn.torch
    q, out = q.t, out.t
    hq = torch.empty(q.numel(), dtype=torch.float64, pin_memory=True)
    ho = torch.empty(out.numel(), dtype=torch.float64, pin_memory=True)
    dq = torch.empty_like(q)
    stream = torch.cuda.current_stream()
    res = {}
    for name, dst, src in (("query_h2d_ms", dq, hq), ("scores_d2h_ms", ho, out)):
        dst.copy_(src, non_blocking=True)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for _ in range(5):
            dst.copy_(src, non_blocking=True)
        ev1.record(stream)
        torch.cuda.synchronize()
        res[name] = round(ev0.elapsed_time(ev1) / 5, 4)
    res["query_bytes"] = 8 * q.numel()
    res["scores_bytes"] = 8 * out.numel()
    return res


def copy_peak_GBs(bn):
    """Measured HBM stream-copy rate: a 1 GiB device-to-device copy, read + write bytes over
    its event-timed duration (mean of 5 after one warm-up)."""
    torch = bn.torch
    src = torch.empty(1 << 27, dtype=torch.float64, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1.0)
    dst.copy_(src)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(5):
        dst.copy_(src)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / 5
    del src, dst
    return round(2 * 8 * (1 << 27) / (ms * 1e-3) / 1e9, 1)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def run_enc_level(bn, args, level):
    """The rerank level against an encrypted database: every diagonal of every block is a
    ciphertext (the paper's deployment stores encrypted rows), enrolled at `level` primes;
    the query is dropped to that level and scored ct x ct with one relinearisation per
    (block, giant step)."""
    w, fa, torch = bn.w, bn.fa, bn.torch
    top = bn.ctx
    ctx = top.at_level(level) if level < w.L else top
    X, centers = bn.wl.candidate_rows(w)
    S = w.slots
    t = time.time()
    blocks = []
    for b in range(w.n_blocks):
        pts = ctx.encode_db_block(X[b * S:(b + 1) * S], w.d, fa.LAYOUT_DIAG, w.B)
        a, e = bn.wl.db_enc_randomness(w, ctx.primes[:ctx.L], 0, w.d, block=b)
        blocks.append(ctx.encrypt_pts(pts, w.d, a, e))
        del pts, a, e
    torch.cuda.synchronize()
    log(f"[bench] encrypted {w.n_blocks} blocks, {w.n_blocks * w.d} ciphertexts at {ctx.L} primes "
        f"({time.time() - t:.1f}s)")
    qv = bn.wl.query_vectors(w, 1, centers)[0]
    q_top = bn.encrypt(pad(qv, w.d))
    q = ctx.new_ct() if ctx is not top else q_top
    out = ctx.new_ct(w.n_blocks)
    ws = ctx.workspace(fa.OP_SCORE_ENC, w.n_blocks, w.d, w.B)

    def step():
        if ctx is not top:
            top.drop_level(ctx, q_top, out=q)
        ctx.score_block(q, blocks, w.d, fa.LAYOUT_DIAG_ENC, w.B, out=out, ws=ws)

    ms = bn.timed(step, args.steps, args.warmup)
    ph = bn.phases(step, ctx)
    err = None
    if not args.no_check:
        err = 0.0
        W_ = ctx.ct_words
        for b in range(w.n_blocks):
            rows = X[b * S:(b + 1) * S].astype(np.float64)
            z = ctx.decode(ctx.decrypt(out[b * W_:(b + 1) * W_]), 80)
            err = max(err, float(np.max(np.abs(z[:len(rows)] - rows @ qv))))
    ptw = ctx.L * w.n
    stream_bytes = 8 * w.n_blocks * w.d * 2 * ptw
    # the encrypted diagonals once, each baby rotation once (the pair chunks of a launch share it
    # through L2), the three-component accumulators written once
    mac_bytes = stream_bytes + 8 * (w.B * 2 * ptw + w.n_blocks * w.G * 3 * ptw)
    res = {"scoring_level_primes": ctx.L, "ms_per_level": round(ms, 4), "value": round(w.rows / (ms * 1e-3), 1),
           "unit": "scores/s", "phases_ms": {"baby_ms": round(ph["baby_ms"], 4),
                                             "mac_ct_ms": round(ph["mac_ms"], 4),
                                             "relin_and_giant_ms": round(ph["giant_ms"], 4)},
           "database_bytes": stream_bytes, "level_hbm_floor_ms": round(stream_bytes / (HBM_PEAK_GBS * 1e9) * 1e3, 4),
           "mac_achieved_GBs": round(mac_bytes / (ph["mac_ms"] * 1e-3) / 1e9, 1), "max_abs_score_err": err,
           "roofline": roofline_of("k_mac_diag_ct", mac_bytes, ph["mac_ms"]),
           "cpu_baseline": None if args.no_cpu_baseline else cpu_baseline_diag(bn, X, qv, L=ctx.L, enc=True)}
    del blocks
    torch.cuda.empty_cache()
    return res


def run_membership(bn, args):
    """The face membership scan (section 3.1, "Membership search"): per step one encrypted 512-d
    query (scale 2^50, 12 primes) is projected to R = 128 under encryption, rescaled, scored
    against all 222,049 centroids enrolled at 11 primes, and every candidate's decision
    cos >= tau is evaluated under encryption (|q_R|^2 by square and fold, tau |q_R| by the
    degree-7 Chebyshev series, two sign steps; levels 12 -> 2).  Its own context and keys."""
    fa, torch, wl = bn.fa, bn.torch, bn.wl
    w = wl.WORKLOADS["face"]
    x = w.extra
    ls = x["log_scale"]
    t = time.time()
    ctx = fa.Context(w.log_n, w.L, w.K, ls)
    s = wl.secret(w)
    ctx.set_secret(s)
    steps = wl.rotation_steps(w)
    ctx.keygen_relin(s, *wl.relin_randomness(w, ctx.primes, ctx.dnum))
    for i in range(0, len(steps), 8):
        chunk = steps[i:i + 8]
        rand = [wl.key_randomness(w, r, ctx.primes, ctx.dnum) for r in chunk]
        ctx.keygen(s, chunk, np.stack([v[0] for v in rand]), np.stack([v[1] for v in rand]))
    levels = [ctx] + [ctx.at_level(l) for l in range(w.L - 1, 1, -1)]
    c11 = levels[1]
    W = wl.projection(w)
    R, B, Bp, S, nb = w.d, w.B, w.B_proj, w.slots, w.n_blocks
    wpts = ctx.encode_projection(W.astype(np.float32), Bp)
    Xr = wl.projected_rows(w, W)
    blocks = [c11.encode_db_block(Xr[i * S:(i + 1) * S].astype(np.float32), R, fa.LAYOUT_DIAG, B)
              for i in range(nb)]
    qs, ids = wl.face_queries(w, 1)
    q = qs[0]
    a, e = wl.enc_randomness(w, ctx.primes[:w.L])
    ct = ctx.encrypt(ctx.encode(np.tile(q, S // w.d_in), ls), a, e)
    coeffs = fa.cheb_fit_sqrt(x["tau"], x["y_lo"], x["y_hi"], x["degree"])
    s_q = 2.0 ** (2 * ls) / ctx.primes[w.L - 1]
    qr, q11, out = ctx.new_ct(), c11.new_ct(), c11.new_ct(nb)
    ws_p = ctx.workspace(fa.OP_PROJECT, 1, R, Bp)
    ws_r = torch.empty(2 * w.L * w.n + 32, dtype=torch.float64, device="cuda")
    ws_m = fa.membership_workspace(c11, nb, R, B, x["degree"])
    torch.cuda.synchronize()
    log(f"[bench] face: keys, {len(levels)} levels, {nb} blocks of {R} diagonals at {c11.L} primes "
        f"({time.time() - t:.1f}s)")
    res_m = {}

    def project():
        ctx.project_ct(ct, wpts, w.d_in, R, Bp, out=qr, ws=ws_p)
        ctx.rescale(c11, qr, out=q11, ws=ws_r)

    def scan():
        res_m["r"] = fa.membership(levels, q11, c11.L, s_q, blocks, R, B, x["y_lo"], x["y_hi"], coeffs, x["m"],
                                   x["iters"], out=out, ws=ws_m)

    def step():
        project()
        scan()

    ms = bn.timed(step, args.steps, args.warmup)
    ms_proj = bn.timed(project, args.steps, 1)
    ms_scan = bn.timed(scan, args.steps, 1)
    c11.profile(True)  # events around the scoring inside the scan (baby, MAC, giant phases)
    scan()
    ph = c11.profile_read()
    sb, sm, sg, st = (ph[k] for k in ("baby_ms", "mac_ms", "giant_ms", "total_ms"))
    c11.profile(False)
    _, L, sc, mo = res_m["r"]
    res = {"workload": w.desc, "ms_per_query": round(ms, 4), "value": round(w.rows / (ms * 1e-3), 1),
           "unit": "decisions/s", "phases_ms": {"project_and_rescale_ms": round(ms_proj, 4),
                                                "scan_ms": round(ms_scan, 4),
                                                "scan_profiled_once": {"score_baby_ms": round(sb, 4),
                                                                       "score_mac_ms": round(sm, 4),
                                                                       "score_giant_ms": round(sg, 4),
                                                                       "score_total_ms": round(st, 4)}},
           "levels": f"{w.L} -> {L}", "tau": x["tau"], "chebyshev_degree": x["degree"],
           "sign_steps": x["iters"], "database_bytes": 8 * nb * R * c11.L * w.n,
           "paper_warm_latency_s_context": 7.0,
           "roofline": roofline_of(MAC_KERNEL, mac_batch_bytes(1, nb * (R // B), B, c11.L * w.n), sm),
           "cpu_baseline": None if args.no_cpu_baseline else cpu_baseline_membership(bn, w, s, q, Xr)}
    if not args.no_check:
        ctw = c11.ct_words
        c2 = levels[w.L - L]
        z = np.concatenate([c2.decode(c2.decrypt(c2.wrap(out.t[i * ctw:i * ctw + 2 * L * c2.n], 2, 1, 0)), ls)
                            for i in range(nb)])
        z = z[:w.rows] * (2.0 ** ls / sc) / mo
        qR = W.astype(np.float32).astype(np.float64).T @ q
        Xm = Xr.astype(np.float32).astype(np.float64)
        y = float(qR @ qR)
        u = (2 * y - x["y_lo"] - x["y_hi"]) / (x["y_hi"] - x["y_lo"])
        tq = float(np.polynomial.chebyshev.chebval(u, coeffs))
        v = (Xm @ qR - tq) / x["m"]
        for _ in range(x["iters"]):
            v = (3 * v - v ** 3) / 2
        margin = Xm @ qR - x["tau"] * np.sqrt(y)
        ok = np.abs(margin) > abs(tq - x["tau"] * np.sqrt(y)) + 1e-4
        res.update({"max_abs_err_vs_float64": float(np.max(np.abs(z - v))),
                    "decision_mismatches": int(np.count_nonzero(np.sign(z[ok]) != np.sign(margin[ok]))),
                    "matches": np.flatnonzero(z > 0).tolist(), "query_identity": int(ids[0])})
    del blocks, levels
    torch.cuda.empty_cache()
    return res


def cpu_baseline_membership(bn, w, s, q, Xr):
    """The oracle timed on a bounded sample of the face scan, extrapolated to one query:
    one rotation at 12 and at 11 primes, the block product with 1 and 2 giant groups on
    block 0 at 11 primes, a relinearised product and rescale at 10 and at 5 primes; then
    (B_proj-1) + (G_proj-1) + 2 rotations for the projection, B-1 baby rotations, the blocks'
    products, log2(d) fold rotations, degree-1 Chebyshev products and 2 * iters sign products
    per block."""
    from oracle import ckks
    x = w.extra
    t_start = time.time()
    top = ckks.Params(logn=w.log_n, L=w.L, K=w.K, log_scale=x["log_scale"])

    def level(L):
        par = top if L == w.L else ckks.Params(logn=w.log_n, L=L, K=w.K, log_scale=x["log_scale"],
                                               primes=top.q[:L] + top.p)
        idx = list(range(L)) + list(range(w.L, w.L + w.K))
        orc = ckks.Oracle(par)

        def key(r):
            a, e = bn.wl.key_randomness(w, r, top.primes, top.dnum)
            return a[:par.dnum][:, idx], e[:par.dnum]
        return par, orc, key

    def enc(par, orc):
        a, e = bn.wl.enc_randomness(w, top.q)
        m = ckks.encode(ckks.replicate(q, par.slots), par.n, x["log_scale"])
        return orc.encrypt(m, np.ascontiguousarray(a[:par.L]), e, s)

    def t_rot(L):
        par, orc, key = level(L)
        k1 = orc.keygen(s, 1, *key(1))
        ct = enc(par, orc)
        t = time.time()
        orc.rotate(ct, 1, k1)
        return time.time() - t, par, orc, key, ct

    def t_mul(L):
        par, orc, key = level(L)
        rlk = orc.keygen_relin(s, *key(0))
        ct = enc(par, orc)
        t = time.time()
        orc.rescale(orc.mul(ct, ct, rlk))
        return time.time() - t

    r12 = t_rot(w.L)[0]
    r11, par, orc, key, ct = t_rot(w.L - 1)
    B, G, nb = w.B, w.d // w.B, w.n_blocks
    keys = {gB: orc.keygen(s, gB, *key(gB)) for gB in (B,)}
    diags = ckks.diagonals(Xr[:par.slots], par.slots, w.d)
    pts = np.stack([ckks.encode_residues(np.roll(diags[gg * B + b], gg * B), par)
                    for gg in range(2) for b in range(B)]).reshape(2, B, par.L, par.n)
    qrot = np.repeat(ct[None], B, axis=0)
    t = time.time()
    orc.bsgs_block(qrot, pts[:1], B, 1, keys)
    g1 = time.time() - t
    t = time.time()
    orc.bsgs_block(qrot, pts, B, 2, keys)
    g2 = time.time() - t
    m10, m5 = t_mul(w.L - 2), t_mul(5)
    Gp = w.d // w.B_proj
    est = ((w.B_proj - 1) + (Gp - 1) + 2) * r12 + (B - 1) * r11 + nb * (g1 + (G - 1) * max(g2 - g1, 0.0)) \
        + int(np.log2(w.d)) * r11 + (1 + x["degree"] - 1) * m10 + nb * 2 * x["iters"] * m5
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    log(f"[bench] oracle sample (face scan): rot {r12:.2f}/{r11:.2f}s, G1 {g1:.2f}s, G2 {g2:.2f}s, "
        f"mul {m10:.2f}/{m5:.2f}s -> query {est:.1f}s ({time.time() - t_start:.1f}s wall)")
    return {"value": round(w.rows / est, 2), "unit": "decisions/s", "cores": cores, "kind": "oracle",
            "sample": "rotations at 12 and 11 primes, the block product with 1 and 2 giant groups on block 0, "
                      "products at 10 and 5 primes; extrapolated to the projection, the scan's scoring, the "
                      "norm's fold, the Chebyshev series and the sign steps of one query",
            "query_s_est": round(est, 2), "cpu_model": cpu_model()}


def roofline_of(kernel, nbytes, ms):
    """The roofline object of a multiply-accumulate kernel: algorithmic bytes over its
    event-timed duration against the 8 TB/s HBM peak (no counter run behind it: traffic null)."""
    achieved = nbytes / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": kernel,
            "algorithmic_bytes": int(nbytes), "avg_ms": round(ms, 4)}


def mac_batch_bytes(nq, n_pairs, B, ptw):
    """Algorithmic bytes of the multiply-accumulate launches for nq queries, following the
    launcher's grouping (4, then 2, then 1 queries per plaintext pass; the full chunks of a
    group's pairs in one launch whose chunks share the rotated queries through L2, a narrower
    launch for the rest): every plaintext once per group, each query's rotations once per
    launch, the accumulators once."""
    total, j = 0, 0
    while j < nq:
        m = 4 if nq - j >= 4 else 2 if nq - j >= 2 else 1
        wide = 32 // m
        p0 = launches = 0
        while p0 < n_pairs:
            left = n_pairs - p0
            p0 += (left // wide) * wide if left >= wide else 16 if (wide > 16 and left > 8) else 8
            launches += 1
        total += n_pairs * B * ptw + launches * m * B * 2 * ptw + m * n_pairs * 2 * ptw
        j += m
    return 8 * total


def run_batch_level(bn, args, r, nq):
    """Cross-query batching on the level r was timed on (same context and resident blocks):
    per step, nq fresh queries are (dropped and) prepared together -- their baby rotations,
    each step's key switches issued for all of them at once -- and then scored together,
    every plaintext pass serving up to four of them."""
    w, fa, torch = bn.w, bn.fa, bn.torch
    top, ctx, blocks = bn.ctx, r["ctx"], r["blocks"]
    X, S = r["X"], w.slots
    qvs = bn.wl.query_vectors(w, nq + 1, r["centers"])[1:]
    q_tops = [bn.encrypt(pad(v, w.d), tag=100 + j) for j, v in enumerate(qvs)]
    qs = [ctx.new_ct() for _ in range(nq)] if ctx is not top else q_tops
    preps = [ctx.new_prep(w.B) for _ in range(nq)]
    outs = [ctx.new_ct(w.n_blocks) for _ in range(nq)]
    ws_p = ctx.prepare_batch_workspace(nq, w.B)
    ws_b = ctx.batch_workspace(nq, w.n_blocks, w.d, w.B)
    stream = torch.cuda.current_stream()
    marks = []

    def step():
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record(stream)
        if ctx is not top:
            for j in range(nq):
                top.drop_level(ctx, q_tops[j], out=qs[j])
        ctx.prepare_batch(qs, w.B, outs=preps, ws=ws_p)
        e1.record(stream)
        ctx.score_batch(qs, preps, blocks, w.d, w.B, outs=outs, ws=ws_b)
        e2.record(stream)
        marks.append((e0, e1, e2))

    ms = bn.timed(step, args.steps, args.warmup)
    torch.cuda.synchronize()
    prep_ms = float(np.mean([a.elapsed_time(b) for a, b, _ in marks[args.warmup:]]))
    score_ms = float(np.mean([b.elapsed_time(c) for _, b, c in marks[args.warmup:]]))
    ph = bn.phases(step, ctx)
    mac_ms = ph["mac_ms"]
    giant_ms = ph["giant_ms"]
    err = None
    if not args.no_check:
        err = 0.0
        W_ = ctx.ct_words
        for j in range(nq):
            for b in range(w.n_blocks):
                rows = X[b * S:(b + 1) * S].astype(np.float64)
                z = ctx.decode(ctx.decrypt(outs[j][b * W_:(b + 1) * W_]), 80)
                err = max(err, float(np.max(np.abs(z[:len(rows)] - rows @ qvs[j]))))
    ptw = ctx.L * w.n
    mac_bytes = mac_batch_bytes(nq, w.n_blocks * w.G, w.B, ctx.L * w.n)
    return {"queries": nq, "scoring_level_primes": ctx.L, "ms_per_step": round(ms, 4),
            "ms_per_query_level": round(ms / nq, 4), "value": round(nq * w.rows / (ms * 1e-3), 1),
            "unit": "scores/s", "phases_ms": {"prepare_ms": round(prep_ms, 4), "score_batch_ms": round(score_ms, 4),
                                              "mac_ms": round(mac_ms, 4), "giant_ms": round(giant_ms, 4)},
            "mac_achieved_GBs": round(mac_bytes / (mac_ms * 1e-3) / 1e9, 1), "mac_algorithmic_bytes": mac_bytes,
            "roofline": roofline_of("k_mac_diag", mac_bytes, mac_ms), "max_abs_score_err": err}


def run_tiny(bn, args):
    w, ctx, fa = bn.w, bn.ctx, bn.fa
    X, _ = bn.wl.candidate_rows(w)
    pts = ctx.encode_db_block(X, w.d, fa.LAYOUT_ROW)
    per = w.slots // w.d
    n_pts = -(-w.rows // per)
    PW = ctx.pt_words
    blocks = [pts[i * PW:(i + 1) * PW] for i in range(n_pts)]
    qv = bn.wl.query_vectors(w)[0]
    q = bn.encrypt(qv)
    out = ctx.new_ct(n_pts)
    ws = ctx.workspace(fa.OP_ROTATE_SUM, n_pts)
    steps = int(np.log2(w.d))

    def step():
        ctx.score_block(q, blocks, w.d, fa.LAYOUT_ROW, 1, out=out)
        ctx.rotate_sum(out, n_pts, 1, steps, ws=ws)

    ms = bn.timed(step, args.steps, args.warmup)
    err = None
    if not args.no_check:
        sc = np.concatenate([bn.decode(out, i, 80)[::w.d] for i in range(n_pts)])[:w.rows]
        err = float(np.max(np.abs(sc - X.astype(np.float64) @ qv)))
    return dict(ms=ms, scores=w.rows, phases={}, err=err, mac_bytes=None, stream_bytes=8 * n_pts * w.L * w.n,
                cpu=(lambda: cpu_baseline_rows(bn, X, qv, n_pts, steps)))


def run_rank(bn, args):
    w, ctx, fa = bn.w, bn.ctx, bn.fa
    W32 = bn.wl.projection(w).astype(np.float32)
    W = W32.astype(np.float64)
    wpts = ctx.encode_projection(W32, w.B_proj)
    Xr = bn.wl.projected_rows(w, W)
    blk = ctx.encode_db_block(Xr.astype(np.float32), w.d, fa.LAYOUT_DIAG, w.B)
    qv = bn.wl.query_vectors(w)[0]
    q = bn.encrypt(qv)
    qr = ctx.new_ct()
    out = ctx.new_ct()
    ws_p = ctx.workspace(fa.OP_PROJECT, 1, w.d, w.B_proj)
    ws_s = ctx.workspace(fa.OP_SCORE, 1, w.d, w.B)
    torch = bn.torch
    stream = torch.cuda.current_stream()
    marks = []

    def step():
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record(stream)
        ctx.project_ct(q, wpts, w.d_in, w.d, w.B_proj, out=qr, ws=ws_p)
        e1.record(stream)
        ctx.score_block(qr, [blk], w.d, fa.LAYOUT_DIAG, w.B, out=out, ws=ws_s)
        e2.record(stream)
        marks.append((e0, e1, e2))

    ms = bn.timed(step, args.steps, args.warmup)
    torch.cuda.synchronize()
    pj = float(np.mean([a.elapsed_time(b) for a, b, _ in marks[args.warmup:]]))
    sc = float(np.mean([b.elapsed_time(c) for _, b, c in marks[args.warmup:]]))
    err = None
    if not args.no_check:
        qR = W.T @ qv
        raw = bn.decode(out, 0, 120)[:w.rows]
        err = float(np.max(np.abs(raw / np.linalg.norm(qR) - Xr @ qR / np.linalg.norm(qR))))
    n_fold = int(np.log2(w.d_in // w.d))
    enc_proj = run_enc_projection(bn, args, wpts, q, W.T @ qv) if args.enc_w else None
    return dict(ms=ms, scores=w.rows, phases={"projection_ms": pj, "scoring_ms": sc}, err=err, mac_bytes=None,
                enc_projection=enc_proj,
                stream_bytes=8 * 2 * w.d * w.L * w.n,
                cpu=(lambda: cpu_baseline_diag(bn, Xr, W.T @ qv, n_blocks=2, n_scores=w.rows,
                                               n_rot=2 * (w.B - 1) + n_fold)))


def run_enc_projection(bn, args, wpts, q, qR):
    """The projection with W's R diagonals encrypted (the paper keeps the projection encrypted on
    the server): R ciphertexts, scored ct x ct with one relinearisation per giant step, then the
    fold.  Timed on its own, after the plaintext-projection step."""
    w, ctx, fa, torch = bn.w, bn.ctx, bn.fa, bn.torch
    a, e = bn.wl.db_enc_randomness(w, ctx.primes[:w.L], 0, w.d, block=99)
    w_cts = ctx.encrypt_pts(wpts, w.d, a, e)
    del a, e
    out = ctx.new_ct()
    ws = ctx.workspace(fa.OP_PROJECT_ENC, 1, w.d, w.B_proj)
    ms = bn.timed(lambda: ctx.project_ct_enc(q, w_cts, w.d_in, w.d, w.B_proj, out=out, ws=ws), args.steps,
                  args.warmup)
    err = None
    if not args.no_check:
        z = bn.decode(out, 0, 80)
        err = float(np.max(np.abs(z - np.tile(qR, w.slots // w.d))))
    res = {"ms_per_projection": round(ms, 4), "max_abs_err_vs_WTq": err,
           "encrypted_diagonals_bytes": 8 * w.d * 2 * w.L * w.n,
           "note": f"Enc(W^T q) with the {w.d} hybrid diagonals of W encrypted ({w.d_in}->{w.d}, baby step "
                   f"{w.B_proj}), ct x ct, one relinearisation per giant step, then the fold"}
    del w_cts
    torch.cuda.empty_cache()
    return res


def topk(sc, k):
    """Ids of the k largest scores, ties to the lower id, in descending order."""
    if k >= len(sc):
        return np.lexsort((np.arange(len(sc)), -sc))
    thr = sc[np.argpartition(-sc, k - 1)[:k]].min()
    above = np.nonzero(sc > thr)[0]
    sel = np.concatenate([above, np.nonzero(sc == thr)[0][:k - len(above)]])
    return sel[np.lexsort((sel, -sc[sel]))]


def run_three_level(bn, args):
    """32 queries, each: coarse level (222,049 rows, 7 blocks) -> client decrypt, top-16 ->
    fine level (2 of 4 fine-pool blocks) -> top-64 -> rerank level (4 of 8 rerank-pool
    blocks, the last truncated to 11,696 rows) -> top-10.  Pool blocks are chosen by
    hashing the kept ids (id mod pool size), deterministic and data-oblivious in cost,
    and passed to the scorer as block ids among the level's resident blocks.  Each
    query is scored at all primes (or dropped to --level primes first) and its baby
    rotations are computed once and reused by the three levels.

    Queries run in groups of --batch (default 4): every query scores all coarse blocks,
    so a group's coarse level is one cross-query batch (one pass over the coarse
    plaintexts per group), and the group's queries are prepared together.  The fine and
    rerank blocks differ per query and are scored one query at a time.  The client's decrypts
    run on a second stream, at the lowest level that holds the scores, so its decode and
    top-k of one query overlap the server's next level on the first; the next group's
    preparation and coarse pass are enqueued before the client takes this group's rerank
    results."""
    w, fa, torch = bn.w, bn.fa, bn.torch
    top_ctx = bn.ctx
    level = args.level if args.level else w.L
    ctx = top_ctx.at_level(level) if level < w.L else top_ctx
    ex = w.extra
    S = w.slots
    nq = args.queries or ex["queries"]
    gq = max(1, min(4, args.batch if args.batch else 1, nq))
    g_coarse, centers = bn.wl.candidate_rows(w, ex["coarse"], stream_extra=1)
    pools = {"coarse": [], "fine": [], "rerank": []}
    rows_of = {"coarse": [], "fine": [], "rerank": []}
    for b in range(-(-ex["coarse"] // S)):
        r = g_coarse[b * S:(b + 1) * S]
        rows_of["coarse"].append(r)
        pools["coarse"].append(ctx.encode_db_block(r, w.d, fa.LAYOUT_DIAG, w.B))
    # the fine and rerank pools are drawn around the same cluster centres
    for name, nb, extra in (("fine", ex["fine_pool_blocks"], 2), ("rerank", ex["rerank_pool_blocks"], 3)):
        X, _ = bn.wl.candidate_rows(w, nb * S, stream_extra=extra, centers=centers)
        for b in range(nb):
            r = X[b * S:(b + 1) * S]
            rows_of[name].append(r)
            pools[name].append(ctx.encode_db_block(r, w.d, fa.LAYOUT_DIAG, w.B))
    torch.cuda.synchronize()
    nblk = sum(len(v) for v in pools.values())
    n_coarse = len(pools["coarse"])
    log(f"[bench] three_level: {nblk} resident blocks at {ctx.L} primes "
        f"({nblk * w.d * ctx.L * w.n * 8 / 1e9:.1f} GB), {gq} queries per coarse pass, {time.time() - bn.t0:.1f}s")
    queries = bn.wl.query_vectors(w, nq, centers)
    qcts = [bn.encrypt(qv, tag=i) for i, qv in enumerate(queries)]
    # two sets of per-query buffers: consecutive groups overlap on the GPU (see below)
    qss = [[ctx.new_ct() for _ in range(gq)] for _ in range(2)] if ctx is not top_ctx else None
    prepss = [[ctx.new_prep(w.B) for _ in range(gq)] for _ in range(2)]
    outs_c = [ctx.new_ct(n_coarse) for _ in range(gq)]
    outs_f = [ctx.new_ct(ex["fine_blocks"]) for _ in range(gq)]
    outs_r = [ctx.new_ct(ex["rerank_blocks"]) for _ in range(gq)]
    ws_p = ctx.prepare_batch_workspace(gq, w.B)
    ws_b = ctx.batch_workspace(gq, n_coarse, w.d, w.B)
    ws_s = ctx.workspace(fa.OP_SCORE_PREPARED, max(ex["fine_blocks"], ex["rerank_blocks"]), w.d, w.B)
    sa = torch.cuda.current_stream()
    sb = torch.cuda.Stream()  # the client's decrypts (default priority)
    # The client decrypts at the lowest level that still holds the scores: the decoder reads
    # only the first primes that cover the scale (2^80) plus 22 bits, and a ciphertext reduced
    # modulo a divisor of Q encrypts the same m + e, so the returned blocks are cut to those
    # primes on the GPU first (fewer limbs to decrypt, transform and copy back; the decoded
    # scores are identical).
    bits, n_dec = 0.0, 0
    while n_dec < ctx.L and bits < 80 + 22:
        bits += math.log2(ctx.primes[n_dec])
        n_dec += 1
    dctx = ctx.at_level(n_dec) if n_dec < ctx.L else ctx
    dbuf = dctx.new_ct(max(n_coarse, ex["fine_blocks"], ex["rerank_blocks"]))
    gpu_ms = []  # per query: [prepare, coarse, fine, rerank]
    errs = []

    from concurrent.futures import ThreadPoolExecutor
    pool = ThreadPoolExecutor(max_workers=8)

    def ev():
        e = torch.cuda.Event(enable_timing=True)
        e.record(sa)
        return e

    def top(ct, nb, k, rows_list, qv, done, n_rows_last=None):
        # client side: wait for the level on the second stream, cut the blocks to the
        # decoder's primes and decrypt them there, then decode the blocks on host threads
        # and keep the top k
        sb.wait_event(done)
        low = ct if dctx is ctx else ctx.drop_level(dctx, ct, out=dbuf.items(0, nb), stream=sb)
        futs = [pool.submit(dctx.decode, dctx.decrypt(low.item(b), stream=sb), 80) for b in range(nb)]
        zs = [f.result() for f in futs]
        scores = []
        for b in range(nb):
            z = zs[b]
            n_valid = len(rows_list[b]) if (b < nb - 1 or n_rows_last is None) else n_rows_last
            scores.append(z[:n_valid])
            if qv is not None:
                ref = rows_list[b][:n_valid].astype(np.float64) @ qv
                errs.append(float(np.max(np.abs(z[:n_valid] - ref))))
        return topk(np.concatenate(scores), k)

    def head(i0, check, slot):
        # server: the group's preparation and its coarse level (one cross-query pass)
        m = min(gq, nq - i0)
        preps = prepss[slot]
        g = {"m": m, "qv": [queries[i0 + j] if check else None for j in range(m)], "qi": [], "preps": preps}
        e0 = ev()
        for j in range(m):
            if qss is not None:
                top_ctx.drop_level(ctx, qcts[i0 + j], out=qss[slot][j])
                g["qi"].append(qss[slot][j])
            else:
                g["qi"].append(qcts[i0 + j])
        ctx.prepare_batch(g["qi"], w.B, outs=preps[:m], ws=ws_p)
        e1 = ev()
        ctx.score_batch(g["qi"], preps[:m], pools["coarse"], w.d, w.B, outs=outs_c[:m], ws=ws_b)
        g["e"] = (e0, e1, ev())
        return g

    def body_fine(g):
        # client top-k of the coarse level, each followed by the server's fine level
        m, qi, qv, preps = g["m"], g["qi"], g["qv"], g["preps"]
        fine = []
        for j in range(m):
            ids = top(outs_c[j], n_coarse, ex["top_coarse"], rows_of["coarse"], qv[j], g["e"][2])
            fsel = sorted(set(int(x) % ex["fine_pool_blocks"] for x in ids))
            fsel = (fsel + [b for b in range(ex["fine_pool_blocks"]) if b not in fsel])[:ex["fine_blocks"]]
            a = ev()
            ctx.score_prepared(qi[j], preps[j], pools["fine"], w.d, w.B, out=outs_f[j], ws=ws_s, block_ids=fsel)
            fine.append((a, ev(), fsel))
        g["fine"] = fine

    def body_rerank(g):
        # client top-k of the fine level, each followed by the server's rerank level
        m, qi, qv, preps, fine = g["m"], g["qi"], g["qv"], g["preps"], g["fine"]
        rer = []
        for j in range(m):
            fsel = fine[j][2]
            ids = top(outs_f[j], len(fsel), ex["top_fine"], [rows_of["fine"][b] for b in fsel], qv[j], fine[j][1])
            rsel = sorted(set(int(x) % ex["rerank_pool_blocks"] for x in ids))
            rsel = (rsel + [b for b in range(ex["rerank_pool_blocks"]) if b not in rsel])[:ex["rerank_blocks"]]
            a = ev()
            ctx.score_prepared(qi[j], preps[j], pools["rerank"], w.d, w.B, out=outs_r[j], ws=ws_s,
                               block_ids=rsel)
            rer.append((a, ev(), rsel))
        g["rer"] = rer

    def tail(g):
        # client top-k of the rerank level; then the group's server time from its events
        m, fine, rer = g["m"], g["fine"], g["rer"]
        for j in range(m):
            rsel = rer[j][2]
            top(outs_r[j], len(rsel), 10, [rows_of["rerank"][b] for b in rsel], g["qv"][j], rer[j][1],
                n_rows_last=ex["rerank_last"])
        rer[-1][1].synchronize()
        e0, e1, e2 = g["e"]
        for j in range(m):
            gpu_ms.append([e0.elapsed_time(e1) / m, e1.elapsed_time(e2) / m, fine[j][0].elapsed_time(fine[j][1]),
                           rer[j][0].elapsed_time(rer[j][1])])

    g0 = head(0, True, 0)  # warm-up group, checked against float64
    body_fine(g0)
    body_rerank(g0)
    tail(g0)
    gpu_ms.clear()
    t = time.time()
    steps = max(1, args.steps)
    starts = [i0 for _ in range(steps) for i0 in range(0, nq, gq)]
    # Groups overlap on the GPU, two deep.  Host order per group k: enqueue group k+1's
    # preparation and coarse pass, take group k's fine results (enqueuing its rerank levels),
    # take group k+1's coarse results (enqueuing its fine levels), take group k's rerank
    # results.  The stream then runs ... fine(k), coarse(k+1), rerank(k), fine(k+1), ... while
    # the client works on earlier results; the two groups in flight use separate query and
    # preparation buffers.
    g = head(starts[0], False, 0)
    body_fine(g)
    for k in range(len(starts)):
        nxt = head(starts[k + 1], False, (k + 1) % 2) if k + 1 < len(starts) else None
        body_rerank(g)
        if nxt is not None:
            body_fine(nxt)
        tail(g)
        g = nxt
    wall = (time.time() - t) / (steps * nq)
    lm = np.array(gpu_ms)
    gpu_q = float(lm.sum(axis=1).mean())
    # the multiply-accumulate launches of one group, timed with the library's phase events
    # (outside the timed queries): the coarse level's batched pass and one rerank level
    ctx.profile(True)
    m = min(gq, nq)
    preps = prepss[0]
    qi = [qcts[j] for j in range(m)] if qss is None else qss[0][:m]
    ctx.prepare_batch(qi, w.B, outs=preps[:m], ws=ws_p)
    ctx.score_batch(qi, preps[:m], pools["coarse"], w.d, w.B, outs=outs_c[:m], ws=ws_b)
    ph_c = ctx.profile_read()
    ctx.score_prepared(qi[0], preps[0], pools["rerank"], w.d, w.B, out=outs_r[0], ws=ws_s,
                       block_ids=list(range(ex["rerank_blocks"])))
    ph_r = ctx.profile_read()
    ctx.profile(False)
    ptw = ctx.L * w.n
    mac_rooflines = {
        "coarse_batch": roofline_of("k_mac_diag", mac_batch_bytes(m, n_coarse * w.G, w.B, ptw), ph_c["mac_ms"]),
        "rerank": roofline_of(MAC_KERNEL, mac_batch_bytes(1, ex["rerank_blocks"] * w.G, w.B, ptw), ph_r["mac_ms"])}
    mac_rooflines["coarse_batch"]["queries_per_pass"] = m
    n_scores = ex["coarse"] + ex["fine_blocks"] * S + (ex["rerank_blocks"] - 1) * S + ex["rerank_last"]
    ph = {"prepare_ms": float(lm[:, 0].mean()), "coarse_ms": float(lm[:, 1].mean()),
          "fine_ms": float(lm[:, 2].mean()), "rerank_ms": float(lm[:, 3].mean()), "query_gpu_ms": gpu_q,
          "query_wall_ms": wall * 1e3}
    blocks_q = n_coarse + ex["fine_blocks"] + ex["rerank_blocks"]
    return dict(ms=gpu_q, scores=n_scores, phases=ph, err=max(errs) if errs else None, mac_bytes=None,
                stream_bytes=8 * blocks_q * w.d * ctx.L * w.n, queries=nq, level=ctx.L, coarse_group=gq,
                mac_rooflines=mac_rooflines,
                cpu=(lambda: cpu_baseline_diag(bn, g_coarse, queries[0], L=ctx.L, n_blocks=blocks_q,
                                               n_scores=n_scores)))


def keyswitch_modmuls(n, L, K, dnum, alpha, B, G, nb):
    """Modular products of the baby and giant phases of one query's level, counted from the
    algorithm (not from the kernels): an NTT or inverse NTT of one limb is (N/2) log2 N butterflies,
    one product each, plus N scalings for an inverse; a fast basis conversion is one product per
    source limb per target word; a key-switch inner product is two per digit per word."""
    import math
    lg = int(math.log2(n))
    ntt = n // 2 * lg            # one forward transform of a limb
    intt = ntt + n               # one inverse transform with its final scaling
    np_ = L + K
    conv_up = dnum * (np_ - alpha)           # converted limbs of one ModUp (alpha sources each)
    modup = L * intt + conv_up * (alpha * n + ntt)
    moddown = 2 * (K * intt + L * (K * n + ntt) + L * n)   # both polynomials, with the P^-1 finish
    # baby: one ModUp of the query, then per rotation the key products over all primes and a ModDown
    baby = modup + (B - 1) * (dnum * np_ * n * 2 + moddown)
    # giant: per (block, giant) pair a ModUp and the key products (plus P c0); one ModDown per block
    pairs = nb * (G - 1)
    giant = pairs * (modup + dnum * np_ * n * 2 + L * n) + nb * moddown
    return baby, giant


def alu_roofline(modmuls, ms, label):
    achieved = modmuls / (ms * 1e-3)
    return {"bound": "alu", "achieved": round(achieved / 1e9, 1), "peak": round(MODMUL_PEAK / 1e9, 1),
            "unit": "Gmodmul/s", "frac": round(achieved / MODMUL_PEAK, 4), "modmuls": int(modmuls),
            "phase": label, "avg_ms": round(ms, 4)}


def measured_traffic(path):
    """HBM bytes per launch of the multiply-accumulate kernel from the committed counter summary, or None
    when the summary is missing or the kernel source changed since it was taken."""
    import hashlib
    import re
    if not path or not os.path.exists(path):
        return None
    txt = open(path).read()
    mb = re.search(r"bytes_per_launch: (\d+)", txt)
    mh = re.search(r"kernel_source_sha256: ([0-9a-f]+)", txt)
    if not mb or not mh:
        return None
    if mac_source_sha256() != mh.group(1):
        return None
    return int(mb.group(1))


LEVEL_TRAFFIC = os.path.join(ROOT, "profiles", "rerank110k_level_traffic.md")


def measured_level_traffic(path=LEVEL_TRAFFIC):
    """Calibrated HBM bytes (FETCH_SIZE + WRITE_SIZE) of every dispatch of one rerank level from the
    committed counter summary, or None when it is missing or the library sources changed since."""
    import re
    from paper_2608_21131_amd.rocprof_summary import sources_sha256
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    got = {k: re.search(rf"{k}: ([0-9a-f]+)", txt) for k in
           ("level_read_bytes", "level_write_bytes", "level_traffic_bytes", "sources_sha256")}
    if not all(got.values()) or got["sources_sha256"].group(1) != sources_sha256():
        return None
    return {k: int(got[k].group(1)) for k in ("level_read_bytes", "level_write_bytes", "level_traffic_bytes")}


MAC_KERNEL = "k_mac_diag3"  # the single-query launches of the rerank level (three steps in flight)


def mac_source_sha256(kernel=MAC_KERNEL):
    """sha256 of the multiply-accumulate kernel's source text (template line to closing brace)."""
    import hashlib
    src = open(os.path.join(ROOT, "paper_2608_21131_amd", "csrc", "fa_kernels.hip")).read()
    a = src.index(f"void {kernel}(")
    a = src.rindex("template <", 0, a)
    b = src.index("\n}\n", a) + 3
    return hashlib.sha256(src[a:b].encode()).hexdigest()


def oracle_at_level(bn, w, L):
    """The oracle's parameters at L ciphertext primes of the workload's chain, and a key
    generator with the workload's key randomness restricted to those primes."""
    from oracle import ckks
    top = ckks.Params(logn=w.log_n, L=w.L, K=w.K)
    par = top if L == w.L else ckks.Params(logn=w.log_n, L=L, K=w.K, primes=top.q[:L] + top.p)
    idx = list(range(L)) + list(range(w.L, w.L + w.K))
    orc = ckks.Oracle(par)

    def rand(r):
        a, e = bn.wl.key_randomness(w, r, top.primes, top.dnum)
        return a[:par.dnum][:, idx], e[:par.dnum]
    return par, orc, rand


def cpu_level_diag(bn, X, qv, L=None):
    """The oracle timed over one whole level of the workload, on the host cores: the B-1
    baby rotations of the query, then every block's product (its d diagonals'
    multiply-accumulate, the giant steps and one ModDown per block), on the workload's
    seeded rows, query and keys.  The keys and each block's integer encoding are prepared
    outside the timed parts; the level time is the sum of the timed parts."""
    from oracle import ckks
    w = bn.w
    B, G, S = w.B, w.G, w.slots
    L = w.L if L is None else L
    t_start = time.time()
    par, orc, rand = oracle_at_level(bn, w, L)
    keys = {r: orc.keygen(bn.s, r, *rand(r)) for r in ckks.steps_for_bsgs(w.d, B)}
    ea, ee = bn.wl.enc_randomness(w, par.q)
    ct = orc.encrypt(ckks.encode(ckks.replicate(pad(qv, w.d), par.slots), par.n, 40), ea, ee, bn.s)
    log(f"[bench] oracle level at {L} primes: {len(keys)} keys ready ({time.time() - t_start:.1f}s)")
    t = time.time()
    qrot = orc.baby_rotations(ct, B, keys)
    t_baby = time.time() - t
    log(f"[bench] oracle level: {B - 1} baby rotations {t_baby:.2f}s")
    t_blocks = []
    for b in range(w.n_blocks):
        rows = np.zeros((min(S, X.shape[0] - b * S), w.d))
        rows[:, :w.dim] = X[b * S:(b + 1) * S]
        c = ckks.layout_b_coeffs(rows, par, w.d, B)
        pts = np.stack([ckks.to_residues(x, par.q) for x in c]).reshape(G, B, par.L, par.n)
        del c
        t = time.time()
        orc.bsgs_block(qrot, pts, B, G, keys)
        t_blocks.append(time.time() - t)
        del pts
        log(f"[bench] oracle level: block {b} ({len(rows)} rows) {t_blocks[-1]:.2f}s")
    level_s = t_baby + sum(t_blocks)
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    log(f"[bench] oracle level at {L} primes: {level_s:.2f}s timed ({time.time() - t_start:.1f}s wall)")
    return {"value": round(w.rows / level_s, 2), "unit": "scores/s", "cores": cores, "kind": "oracle",
            "sample": f"one whole level timed: {B - 1} baby rotations + the products of all {w.n_blocks} blocks "
                      f"({w.rows} rows, {w.n_blocks * w.d} diagonals, B={B}, G={G}) at {L} primes, the same "
                      f"seeded rows, query and keys as the GPU level",
            "level_s": round(level_s, 3), "phases_s": {"baby_rotations": round(t_baby, 3),
                                                        "blocks": [round(x, 3) for x in t_blocks]},
            "cpu_model": cpu_model()}


def run_three_level_field(args):
    """The full three-level query as a field of the default line: its own context (the
    three_level workload's keys), 32 queries back to back at all 12 primes."""
    import copy
    a3 = copy.copy(args)
    a3.workload, a3.baby_step, a3.level, a3.queries = "three_level", 0, 0, 0
    a3.steps = 1
    bn3 = Bench(a3)
    r = run_three_level(bn3, a3)
    w = bn3.w
    ph = r["phases"]
    res = {"workload": w.desc, "queries": r["queries"], "scoring_level_primes": r["level"],
           "queries_per_coarse_pass": r["coarse_group"], "ms_per_query_gpu": round(r["ms"], 4),
           "value": round(r["scores"] / (r["ms"] * 1e-3), 1), "unit": "scores/s",
           "scores_per_query": r["scores"], "phases_ms": {k: round(v, 4) for k, v in ph.items()},
           "with_client": {"query_wall_ms": round(ph["query_wall_ms"], 3),
                           "scores_per_s": round(r["scores"] / (ph["query_wall_ms"] * 1e-3), 1)},
           "query_hbm_floor_ms": round(r["stream_bytes"] / (HBM_PEAK_GBS * 1e9) * 1e3, 4),
           "frac_of_hbm_roofline": round(r["stream_bytes"] / (HBM_PEAK_GBS * 1e9) * 1e3 / r["ms"], 4),
           "max_abs_score_err": r["err"],
           "roofline": r["mac_rooflines"]["coarse_batch"], "mac_rooflines": r["mac_rooflines"],
           "cpu_baseline": None if args.no_cpu_baseline else r["cpu"]()}
    del bn3, r
    import torch
    torch.cuda.empty_cache()
    return res


def cpu_baseline_rows(bn, X, qv, n_pts, steps):
    """The row layout on the oracle: time one plaintext product and two rotations of the same
    parameters and extrapolate to n_pts products, each followed by `steps` rotate-and-sum steps."""
    from oracle import ckks
    w = bn.w
    t_start = time.time()
    par, orc, rand = oracle_at_level(bn, w, w.L)
    keys = {r: orc.keygen(bn.s, r, *rand(r)) for r in (1, 2)}
    ea, ee = bn.wl.enc_randomness(w, par.q)
    ct = orc.encrypt(ckks.encode(ckks.replicate(qv, par.slots), par.n, 40), ea, ee, bn.s)
    pt = ckks.to_residues(ckks.encode(ckks.pack_rows(X.astype(np.float64), par.slots, w.d)[0], par.n, 40), par.q)
    t = time.time()
    orc.mul_plain(ct, pt)
    t_mul = time.time() - t
    t = time.time()
    orc.rotate(ct, 1, keys[1])
    orc.rotate(ct, 2, keys[2])
    t_rot = (time.time() - t) / 2
    est = n_pts * (t_mul + steps * t_rot)
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    log(f"[bench] oracle sample (rows): mul {t_mul:.3f}s, rot {t_rot:.3f}s -> {est:.2f}s "
        f"({time.time() - t_start:.1f}s wall)")
    return {"value": round(w.rows / est, 2), "unit": "scores/s", "cores": cores, "kind": "oracle",
            "sample": f"1 plaintext product + 2 rotations at {w.L} primes; extrapolated to {n_pts} products "
                      f"x (1 + {steps} rotate-and-sum steps)",
            "level_s_est": round(est, 3), "cpu_model": cpu_model()}


def cpu_baseline_diag(bn, X, qv, L=None, enc=False, n_blocks=None, n_scores=None, n_rot=None):
    """Time the oracle on a sample of the same level and scale to scores/s.

    Sample: two rotations of the query, and the oracle's block product with
    G = 1 and G = 2 on the first B diagonals of block 0 (with enc, the diagonals
    encrypted and the ct x ct product with its relinearisations).  Level
    estimate = (B-1) t_rot + n_blocks (t_G1 + (G-1)(t_G2 - t_G1)).  n_blocks,
    n_scores and n_rot (the rotations outside the block products, B-1 by default) override
    the workload's: the three-level query has its baby rotations once, then the
    blocks of all three levels; the rank reduction has two baby-step sets, the
    projection's two fold rotations, and two block products (W's and the
    candidates').
    """
    from oracle import ckks
    w = bn.w
    B, G = w.B, w.G
    L = w.L if L is None else L
    t_start = time.time()
    par, orc, rand = oracle_at_level(bn, w, L)
    keys = {r: orc.keygen(bn.s, r, *rand(r)) for r in (1, 2, B)}
    rlk = orc.keygen_relin(bn.s, *rand(0)) if enc else None
    ea, ee = bn.wl.enc_randomness(w, par.q)
    m = ckks.encode(ckks.replicate(pad(qv, w.d), par.slots), par.n, 40)
    ct = orc.encrypt(m, ea, ee, bn.s)
    t = time.time()
    orc.rotate(ct, 1, keys[1])
    orc.rotate(ct, 2, keys[2])
    t_rot = (time.time() - t) / 2
    S = par.slots
    rows = np.zeros((min(S, X.shape[0]), w.d))
    rows[:, :w.dim] = X[:S]
    diags = ckks.diagonals(rows, S, w.d)
    coeffs = [ckks.encode(np.roll(diags[gg * B + b], gg * B), par.n, 40) for gg in range(2) for b in range(B)]
    pts = np.stack([ckks.to_residues(c, par.q) for c in coeffs]).reshape(2, B, par.L, par.n)
    if enc:
        da, de = bn.wl.db_enc_randomness(w, par.q, 0, 2 * B)
        cts = np.stack([orc.encrypt(c, da[j], de[j], bn.s) for j, c in enumerate(coeffs)])
        cts = cts.reshape(2, B, 2, par.L, par.n)
    qrot = np.repeat(ct[None], B, axis=0)
    t = time.time()
    if enc:
        orc.bsgs_block_ct(qrot, cts[:1], B, 1, keys, rlk)
    else:
        orc.bsgs_block(qrot, pts[:1], B, 1, keys)
    t_g1 = time.time() - t
    t = time.time()
    if enc:
        orc.bsgs_block_ct(qrot, cts, B, 2, keys, rlk)
    else:
        orc.bsgs_block(qrot, pts, B, 2, keys)
    t_g2 = time.time() - t
    nb = w.n_blocks if n_blocks is None else n_blocks
    nr = B - 1 if n_rot is None else n_rot
    est = nr * t_rot + nb * (t_g1 + (G - 1) * max(t_g2 - t_g1, 0.0))
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    log(f"[bench] oracle sample at {L} primes{' (encrypted blocks)' if enc else ''}: rot {t_rot:.2f}s, "
        f"G1 {t_g1:.2f}s, G2 {t_g2:.2f}s -> {nb} blocks {est:.1f}s ({time.time() - t_start:.1f}s wall)")
    return {"value": round((w.rows if n_scores is None else n_scores) / est, 2), "unit": "scores/s", "cores": cores,
            "kind": "oracle",
            "sample": f"2 rotations + {'encrypted ' if enc else ''}block product with 1 and 2 giant groups "
                      f"(B={B}) on block 0 at {L} primes; extrapolated to {nr} rotations and {nb} blocks x "
                      f"{G} groups",
            "level_s_est": round(est, 2), "cpu_model": cpu_model()}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU (the scoring level runs on one MI355X); --gpus {args.gpus} is not "
              "supported", file=sys.stderr)
        sys.exit(2)
    bn = Bench(args)
    w = bn.w
    if w.name == "face":
        m = run_membership(bn, args)
        res = {"metric": "encrypted membership decisions/s + ms/query, 222,049 x 512-dim face centroids at "
                         "R=128, one MI355X",
               "value": m.pop("value"), "unit": m.pop("unit"), "n_gpus": 1, "steps": args.steps,
               "warmup": args.warmup, "ms_per_step": m["ms_per_query"], "higher_is_better": True,
               "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
               "config": {"workload": m.pop("workload"), "log_n": w.log_n, "L": w.L, "K": w.K,
                          "log_scale": w.extra["log_scale"], "d_in": w.d_in, "R": w.d, "baby_step": w.B},
               **m}
        print(json.dumps(res), flush=True)
        return
    runner = {"tiny": run_tiny, "fine": run_diag_level, "rerank": run_diag_level, "rank": run_rank,
              "three_level": run_three_level}[w.name]
    r = runner(bn, args)
    ms = r["ms"]
    value = r["scores"] / (ms * 1e-3)
    log(f"[bench] {w.name}: {ms:.3f} ms/step, {value / 1e6:.2f} M scores/s, phases {r['phases']}, err {r['err']}")
    roofline = None
    if r["mac_bytes"]:
        mac_ms = r["phases"]["mac_ms"]
        achieved = r["mac_bytes"] / (mac_ms * 1e-3) / 1e9
        traffic = measured_traffic(args.traffic) if (w.name == "rerank" and w.B == 64 and not args.level) else None
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic, "kernel": MAC_KERNEL,
                    "algorithmic_bytes": r["mac_bytes"], "avg_ms": round(mac_ms, 4),
                    "measured_copy_GBs": copy_peak_GBs(bn)}
    elif r.get("mac_rooflines"):
        roofline = r["mac_rooflines"]["coarse_batch"]
    cpu = None
    if not args.no_cpu_baseline and r.get("cpu"):
        cpu = r["cpu"]()
        cpu["cpu_model"] = cpu_model()
    floor_ms = r["stream_bytes"] / (HBM_PEAK_GBS * 1e9) * 1e3
    cfg = {"workload": w.desc, "rows_scored_per_step": r["scores"], "d": w.d, "baby_step": w.B,
           "giant_steps": w.G, "log_n": w.log_n, "L": w.L, "K": w.K, "log_scale": 40}
    if args.level and args.level < w.L:
        cfg["scoring_level_primes"] = args.level
        cfg["workload"] += (f"; query dropped to {args.level} ciphertext primes and database enrolled at that "
                            "level before scoring")
    if r.get("queries"):
        cfg["queries_per_step"] = r["queries"]
    if r.get("coarse_group"):
        cfg["queries_per_coarse_pass"] = r["coarse_group"]
    if r.get("level") and r["level"] < w.L:
        cfg["scoring_level_primes"] = r["level"]
    res = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "scores/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "ms_per_level": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": cfg,
        "phases_ms": {k: round(v, 4) for k, v in r["phases"].items()},
        "level_hbm_floor_ms": round(floor_ms, 4),
        "level_frac_of_hbm_roofline": round(floor_ms / ms, 4),
        "level_traffic": None,
        "max_abs_score_err": r["err"],
        "transfers_outside_timing": r.get("io"),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if (w.name in ("rerank", "fine") and not args.level and r["phases"].get("baby_ms")
            and r["phases"].get("giant_ms")):
        # the key-switch phases against the fp64 ALU roofline (modular products per second); the
        # digits hold K primes each (alpha = K), dnum = ceil(L / K)
        dnum = -(-w.L // w.K)
        bmm, gmm = keyswitch_modmuls(w.n, w.L, w.K, dnum, w.K, w.B, w.G, w.n_blocks)
        res["keyswitch_alu"] = {"baby": alu_roofline(bmm, r["phases"]["baby_ms"], "baby rotations"),
                                "giant": alu_roofline(gmm, r["phases"]["giant_ms"], "giant steps")}
    if w.name == "rerank" and w.B == 64 and not args.level:
        lt = measured_level_traffic()
        if lt:
            # every dispatch of one level, counted by rocprofv3 (profiles/rerank110k_level_traffic.md)
            fl = lt["level_traffic_bytes"] / (HBM_PEAK_GBS * 1e9) * 1e3
            res["level_traffic"] = {"bytes": lt["level_traffic_bytes"], "read_bytes": lt["level_read_bytes"],
                                    "write_bytes": lt["level_write_bytes"], "floor_ms": round(fl, 4),
                                    "frac_of_floor": round(fl / ms, 4),
                                    "source": "profiles/rerank110k_level_traffic.md"}
    if r.get("enc_projection"):
        res["enc_projection"] = r["enc_projection"]
    if w.name == "three_level":
        res["metric"] = ("server GPU time per query (3 levels) + aggregate server scores/s, 32 encrypted queries "
                         "back-to-back, one MI355X")
        res["ms_per_level"] = None
        res["mac_rooflines"] = r["mac_rooflines"]
        # the client's part (decrypt, decode, top-k between levels) runs on the host between the
        # levels; the wall clock around whole queries, client included, is reported beside
        ph = r["phases"]
        res["with_client"] = {"query_wall_ms": round(ph["query_wall_ms"], 3),
                              "scores_per_s": round(r["scores"] / (ph["query_wall_ms"] * 1e-3), 1),
                              "note": "wall clock per query over the timed queries, the client's host-side "
                                      "decrypt, decode and top-k between levels included"}
    extra = w.name == "rerank" and not args.level
    r2 = None
    if extra and args.also_level and args.also_level < w.L:
        import copy
        a2 = copy.copy(args)
        a2.level = args.also_level
        r2 = run_diag_level(bn, a2)
        res["level_drop"] = {"scoring_level_primes": args.also_level, "ms_per_level": round(r2["ms"], 4),
                             "value": round(r2["scores"] / (r2["ms"] * 1e-3), 1), "unit": "scores/s",
                             "phases_ms": {k: round(v, 4) for k, v in r2["phases"].items()},
                             "max_abs_score_err": r2["err"],
                             "level_hbm_floor_ms": round(r2["stream_bytes"] / (HBM_PEAK_GBS * 1e9) * 1e3, 4),
                             "mac_achieved_GBs": round(r2["mac_bytes"] / (r2["phases"]["mac_ms"] * 1e-3) / 1e9, 1),
                             "roofline": roofline_of(MAC_KERNEL, r2["mac_bytes"], r2["phases"]["mac_ms"]),
                             "cpu_baseline": None if args.no_cpu_baseline else r2["cpu"]()}
        log(f"[bench] level drop to {args.also_level} primes: {r2['ms']:.3f} ms/level")
    if extra and args.enc_level:
        res["enc_db"] = run_enc_level(bn, args, min(args.enc_level, w.L))
        log(f"[bench] encrypted database at {res['enc_db']['scoring_level_primes']} primes: "
            f"{res['enc_db']['ms_per_level']:.3f} ms/level")
    if extra and args.batch > 1:
        res["query_batch"] = [run_batch_level(bn, args, r, args.batch)]
        if r2 is not None:
            res["query_batch"].append(run_batch_level(bn, a2, r2, args.batch))
        for qb in res["query_batch"]:
            ref = cpu if qb["scoring_level_primes"] == w.L else res.get("level_drop", {}).get("cpu_baseline")
            qb["cpu_baseline"] = None if ref is None else dict(
                ref, sample="the oracle scores a batch's queries one by one: " + ref["sample"])
            log(f"[bench] batch of {qb['queries']} at {qb['scoring_level_primes']} primes: "
                f"{qb['ms_per_query_level']:.3f} ms per query level, {qb['value'] / 1e6:.1f} M scores/s")
    if extra and args.membership:
        res["membership"] = run_membership(bn, args)
        log(f"[bench] face membership scan: {res['membership']['ms_per_query']:.3f} ms per query")
    if extra and args.three_level:
        res["three_level"] = run_three_level_field(args)
        log(f"[bench] three-level query at {res['three_level']['scoring_level_primes']} primes: "
            f"{res['three_level']['ms_per_query_gpu']:.3f} GPU ms per query")
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
