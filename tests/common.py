"""Shared set-up for the GPU parity tests: seeded inputs handed identically to
the library (through the C ABI) and to the CPU oracle."""
from __future__ import annotations

import sys

import numpy as np

from oracle import ckks
from paper_2608_21131_amd import gen

# parameter sets: (log2 N, L, K)
PARAMS = {
    "tiny": (10, 3, 1),
    "tiny1": (10, 3, 3),   # one digit (alpha = K = L)
    "small": (11, 4, 2),
    "p1": (13, 3, 1),
    "p2": (15, 8, 2),
    "p4": (16, 12, 3),
    # short last digits (fewer limbs than alpha) and the remaining transform splits
    "s12": (12, 5, 2),     # digits of 2, 2, 1 primes
    "s14": (14, 7, 4),     # digits of 4, 3 primes
    "d8": (13, 16, 2),     # eight digits, the most the key-switch kernels take
    # the largest parameters the library takes, at the full ring size
    "max8": (16, 16, 2),   # 16 ciphertext primes in eight digits
    "max20": (16, 16, 4),  # 16 + 4: the most primes
}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


class Pair:
    """A library context and an oracle over the same parameters with the same secret."""

    def __init__(self, name: str, wid: int = 0):
        from paper_2608_21131_amd import fa
        logn, L, K = PARAMS[name]
        self.name = name
        self.wid = wid
        self.par = ckks.Params(logn=logn, L=L, K=K)
        self.orc = ckks.Oracle(self.par)
        self.ctx = fa.Context(logn, L, K, 40)
        assert self.ctx.primes == self.par.primes, "prime selection differs"
        self.n = self.par.n
        self.s = gen.ternary_secret(gen.rng(wid, gen.STREAM_SECRET), self.n)
        self.ctx.set_secret(self.s)
        self.okeys = {}

    def key_rand(self, r: int):
        par = self.par
        a = gen.uniform_residues(gen.rng(self.wid, gen.STREAM_KEY_A, r), par.primes, par.dnum, par.n)
        e = gen.rounded_gaussian(gen.rng(self.wid, gen.STREAM_KEY_E, r), (par.dnum, par.n))
        return a, e

    def keys(self, steps, oracle: bool = True):
        steps = sorted(set(int(r) for r in steps))
        new = [r for r in steps if not self.ctx.has_key(r)]
        if new:
            rand = [self.key_rand(r) for r in new]
            a = np.stack([x[0] for x in rand])
            e = np.stack([x[1] for x in rand])
            self.ctx.keygen(self.s, new, a, e)
        if oracle:
            for r in steps:
                if r not in self.okeys:
                    a, e = self.key_rand(r)
                    self.okeys[r] = self.orc.keygen(self.s, r, a, e)
        return self.okeys

    def enc_rand(self, tag: int = 0):
        par = self.par
        a = gen.uniform_residues(gen.rng(self.wid, gen.STREAM_ENC_A, tag), par.q, 1, par.n)[0]
        e = gen.rounded_gaussian(gen.rng(self.wid, gen.STREAM_ENC_E, tag), par.n)
        return a, e

    def encrypt_both(self, m, tag: int = 0):
        a, e = self.enc_rand(tag)
        ct_dev = self.ctx.encrypt(m, a, e)
        ct_orc = self.orc.encrypt(m, a, e, self.s)
        return ct_dev, ct_orc

    def export_ct(self, t, count: int = 1):
        out = self.ctx.export(t, 2 * count)
        return out.reshape(count, 2, self.par.L, self.n)
