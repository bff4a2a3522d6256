"""Host-side model of the Gram jobs of the fit and the probe.

The Gram kernel decodes each job (up to four 128 x 128 blocks P_a^T P_b,
one per wave) from its index; this model replays that decoding for every
job of a launch and checks that each needed block is computed exactly once,
that every plane id and output block index stays inside its array, and that
no job needs more distinct planes than a stage of the kernel's LDS ring
holds (four; key jobs stage each plane's rounding residual beside it)."""

import itertools

import numpy as np
import pytest

MAXPLANES = 4


# the kernel's block order per k: (a, b), b == 4 the target plane
ORDER = {1: [0x00, 0x04],
         2: [0x00, 0x01, 0x04, 0x11, 0x14],
         3: [0x00, 0x01, 0x02, 0x04, 0x11, 0x12, 0x14, 0x22, 0x24],
         4: [0x00, 0x01, 0x02, 0x03, 0x11, 0x12, 0x13, 0x14, 0x22, 0x23, 0x24, 0x04, 0x33, 0x34]}


def lo_slot(H, pid):
    return (pid // (2 * H)) * H + pid % H


def decode(mode, L_s, L_t, H, k, idx, job):
    """Blocks (wave, pa, pb, out, key) of one job, as the kernel decodes them."""
    nsrc = L_s * 2 * H
    if mode == 0:
        nbl = k * (k + 3) // 2
        assert len(ORDER[k]) == nbl
        nch = (nbl + 3) // 4
        task, ch = divmod(job, nch)
        l, hk = task % L_t, task // L_t
        kv, h = hk & 1, hk >> 1
        nblk = min(nbl - 4 * ch, 4)
        blocks = []
        for w in range(nblk):
            e = 4 * ch + w
            a, b = ORDER[k][e] >> 4, ORDER[k][e] & 15
            pa = (int(idx[l][a]) * 2 + kv) * H + h
            if b == 4:
                pb = nsrc + (l * 2 + kv) * H + h
                key = ("xy", l, h, kv, a)
            else:
                pb = (int(idx[l][b]) * 2 + kv) * H + h
                key = ("xx", l, h, kv, a, b)
            blocks.append((w, pa, pb, task * nbl + e, key))
        return kv, blocks
    n_sp, n_lp = (L_s + 1) // 2, (L_t + 1) // 2
    per = n_sp * n_lp + (L_s + 3) // 4
    grp, c = divmod(job, per)
    h, kv = grp >> 1, grp & 1
    base = L_s * (2 * h + kv)
    blocks = []
    if c < n_sp * n_lp:
        fb = n_sp // 4
        if c < fb * 4 * n_lp:
            sbk, rem, rows = c // (4 * n_lp), c % (4 * n_lp), 4
        else:
            sbk, rem, rows = fb, c - fb * 4 * n_lp, n_sp - fb * 4
        lp, r = divmod(rem, rows)
        sp = sbk * 4 + r
        for w in range(4):
            s_, l = 2 * sp + (w >> 1), 2 * lp + (w & 1)
            if s_ >= L_s or l >= L_t:
                continue
            blocks.append((w, (s_ * 2 + kv) * H + h, nsrc + (l * 2 + kv) * H + h,
                           (base + s_) * (L_t + 1) + 1 + l, ("pq", s_, l, h, kv)))
    else:
        c2 = c - n_sp * n_lp
        for w in range(4):
            s_ = 4 * c2 + w
            if s_ >= L_s:
                continue
            p = (s_ * 2 + kv) * H + h
            blocks.append((w, p, p, (base + s_) * (L_t + 1), ("self", s_, h, kv)))
    return kv, blocks


def planes_of(blocks):
    return {p for _, pa, pb, _, _ in blocks for p in (pa, pb)}


def n_jobs(mode, L_s, L_t, H, k):
    if mode == 0:
        nbl = k * (k + 3) // 2
        return L_t * H * 2 * ((nbl + 3) // 4)
    return H * 2 * (((L_s + 1) // 2) * ((L_t + 1) // 2) + (L_s + 3) // 4)


@pytest.mark.parametrize("k", [1, 2, 3, 4])
@pytest.mark.parametrize("shape", [(40, 64, 8), (5, 3, 2), (1, 1, 1)])
def test_fit_jobs_cover_each_block_once(k, shape):
    L_s, L_t, H = shape
    if k > L_s:
        pytest.skip("k > L_s")
    rng = np.random.default_rng(k)
    idx = np.stack([rng.choice(L_s, k, replace=False) for _ in range(L_t)])
    P = (L_s + L_t) * 2 * H
    nbl = k * (k + 3) // 2
    seen, outs = set(), set()
    for job in range(n_jobs(0, L_s, L_t, H, k)):
        kv, blocks = decode(0, L_s, L_t, H, k, idx, job)
        assert 1 <= len(blocks) <= 4
        assert len(planes_of(blocks)) <= MAXPLANES
        for w, pa, pb, out, key in blocks:
            assert 0 <= pa < P and 0 <= pb < P
            assert kv == 1 or 0 <= P + lo_slot(H, pa) < P + P // 2
            assert 0 <= out < L_t * H * 2 * nbl
            assert key not in seen and out not in outs
            seen.add(key)
            outs.add(out)
    want = {("xx", l, h, kv, a, b) for l, h, kv in itertools.product(range(L_t), range(H), range(2))
            for a in range(k) for b in range(a, k)}
    want |= {("xy", l, h, kv, a) for l, h, kv in itertools.product(range(L_t), range(H), range(2))
             for a in range(k)}
    assert seen == want
    assert outs == set(range(L_t * H * 2 * nbl))


@pytest.mark.parametrize("shape", [(40, 64, 8), (5, 3, 2), (2, 7, 1), (9, 1, 1), (1, 1, 1)])
def test_probe_jobs_cover_each_block_once(shape):
    L_s, L_t, H = shape
    P = (L_s + L_t) * 2 * H
    seen, outs = set(), set()
    for job in range(n_jobs(1, L_s, L_t, H, 1)):
        kv, blocks = decode(1, L_s, L_t, H, 1, None, job)
        assert 1 <= len(blocks) <= 4
        assert len(planes_of(blocks)) <= MAXPLANES
        for w, pa, pb, out, key in blocks:
            assert 0 <= pa < P and 0 <= pb < P and 0 <= out < L_s * H * 2 * (L_t + 1)
            assert key[-1] == kv
            assert key not in seen and out not in outs
            seen.add(key)
            outs.add(out)
    assert len(seen) == L_s * H * 2 * (L_t + 1)
    assert outs == set(range(L_s * H * 2 * (L_t + 1)))


def test_probe_jobs_share_planes_across_an_xcd():
    """32 consecutive cross jobs (the CUs of one XCD) touch 8 source and 16
    target planes on the Qwen3-14B->32B shape."""
    L_s, L_t, H = 40, 64, 8
    for start in (0, 32, 96):
        planes = set()
        for job in range(start, start + 32):
            planes |= planes_of(decode(1, L_s, L_t, H, 1, None, job)[1])
        assert len(planes) == 24


def test_matches_library_job_count():
    """The library's workspace sizes imply the same block counts."""
    from paper_2608_03893_amd import kvx
    d = kvx.Dims(L_s=40, L_t=64, H=8, T=32768, d=128, k=4)
    Npad, P = 32768, (40 + 64) * 2 * 8
    up = lambda n: (n + 255) // 256 * 256
    base = up(32768 * 128 * 12) + up((P + P // 2) * 128 * Npad * 2) + 2 * up(P * 128 * 8)
    fit_blocks = 64 * 8 * 2 * 14
    assert kvx.fit_workspace_bytes(d) == (base + up(fit_blocks * 128 * 128 * 4)
                                          + up(64 * 8 * 2 * 512 * 512 * 8)
                                          + up(64 * 8 * 2 * 512 * 128 * 8))
    assert kvx.probe_workspace_bytes(d) == base + up(40 * 8 * 2 * 65 * 128 * 128 * 4)
    assert kvx.fit_workspace_bytes(kvx.Dims(L_s=4, L_t=3, H=2, T=0, d=128, k=2)) == 0
    assert kvx.fit_workspace_bytes(kvx.Dims(L_s=4, L_t=3, H=2, T=64, d=64, k=2)) == 0
    assert kvx.fit_workspace_bytes(kvx.Dims(L_s=4, L_t=3, H=2, T=64, d=128, k=5)) == 0
