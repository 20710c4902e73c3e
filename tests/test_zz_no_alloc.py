"""fa_rotate_static, the rotation for callers that cannot allocate: its key-switch scratch
lives in the library's fixed device array instead of a caller workspace.  Through the C ABI
it must write exactly what fa_rotate writes (bit-exact, so also the oracle's rotation), on
consecutive calls of different sizes that reuse the array, and refuse a context whose
rotation needs more scratch than the array holds."""
import numpy as np
import pytest

from oracle import ckks
from paper_2608_21131_amd import gen

from common import Pair, say

pytestmark = pytest.mark.gpu


def _rotate_both(p, r, tag):
    v = np.random.default_rng(tag).uniform(-1, 1, p.par.slots)
    ct, ct_o = p.encrypt_both(ckks.encode(v, p.n, 40), tag=tag)
    keys = p.keys([r], oracle=p.n <= 2048)
    say(f"[static] {p.name}: rotation by {r}, fixed scratch vs workspace")
    got = p.ctx.export(p.ctx.rotate_static(ct, r)).reshape(2, p.par.L, p.n)
    ref = p.ctx.export(p.ctx.rotate(ct, r)).reshape(2, p.par.L, p.n)
    assert np.array_equal(got, ref)
    if p.n <= 2048:
        assert np.array_equal(got, p.orc.rotate(ct_o, r, keys[r]))
    # meaning: the rolled slots, within one key switch's noise (the extended digits are kept
    # canonical, not centred: up to about 1e-4 per slot at N = 2^16 over a full random vector)
    z = p.ctx.decode(p.ctx.decrypt(p.ctx.rotate_static(ct, r)), 40)
    assert np.max(np.abs(z - np.roll(v, -r))) < 1e-3


def test_static_scratch_rotation_matches_workspace_rotation():
    # the largest supported rotation first (N=2^16, 12+3 primes: 63 MiB of scratch), then a
    # smaller one that finds the array holding the previous call's contents
    big = Pair("p4", wid=40)
    _rotate_both(big, 5, 40)
    small = Pair("tiny", wid=41)
    _rotate_both(small, 3, 41)
    _rotate_both(big, 7, 42)


def test_static_scratch_refuses_a_rotation_larger_than_the_array():
    from paper_2608_21131_amd import fa
    ctx = fa.Context(16, 16, 2, 40)  # 8 digits over 18 primes: 114 MiB of rotation scratch
    assert ctx.workspace_bytes(fa.OP_ROTATE, 1) > (64 << 20)
    s = gen.ternary_secret(gen.rng(43, gen.STREAM_SECRET), ctx.n)
    ctx.set_secret(s)
    ct = ctx.new_ct().zero_()
    ct.log_scale = 40
    with pytest.raises(fa.FaError) as ei:
        ctx.rotate_static(ct, 1)
    assert ei.value.code == fa.FA_E_NOMEM and "fixed array" in str(ei.value)
