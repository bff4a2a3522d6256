"""Host-side models of the Gram jobs of the fit and the probe.

The Gram kernel decodes each job (up to four 128 x 128 blocks P_a^T P_b,
one per wave) from its index.  The probe's jobs follow from arithmetic on the
job index; the fit's come from its block plan, a function of the index table
alone: each distinct pair of source layers is computed once per (head, K|V),
by the first target layer whose list holds it, and each target layer's cross
blocks and owned pairs are packed first-fit into jobs.  These models replay
both and check that each needed block is computed exactly once, that every
plane id and output block index stays inside its array, that no job needs
more distinct planes than a stage of the kernel's LDS ring holds (four; key
jobs stage each plane's rounding residual beside it), and that the solve
finds every block of its design Gram, in the right orientation."""

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


def plan_layer(idx, k, l):
    """Items of target layer l (cross blocks ("x", a, l) of its distinct
    sources, then the pairs ("p", a, b) it owns) and the job of each item."""
    s = [int(v) for v in idx[l]]
    items = [("x", s[i], l) for i in range(k) if s[i] not in s[:i]]
    for i in range(k):
        for j in range(i, k):
            a, b = s[i], s[j]
            seen = any(a in list(idx[l2]) and b in list(idx[l2]) for l2 in range(l))
            seen = seen or any({s[i2], s[j2]} == {a, b} and (i2, j2) < (i, j)
                               for i2 in range(k) for j2 in range(i2, k))
            if not seen:
                items.append(("p", a, b))
    job = [None] * len(items)
    n_jobs = 0
    while None in job:
        planes, cnt = set(), 0
        for t, it in enumerate(items):
            if job[t] is not None or cnt == 4:
                continue
            pl = {it[1], "Q"} if it[0] == "x" else {it[1], it[2]}
            if len(planes | pl) > 4:
                continue
            planes |= pl
            job[t] = n_jobs
            cnt += 1
        n_jobs += 1
    return items, job, n_jobs


_PLANS = {}


def fit_plan(idx, k):
    key = (np.asarray(idx).tobytes(), np.asarray(idx).shape, k)
    if key not in _PLANS:
        _PLANS[key] = _fit_plan(idx, k)
    return _PLANS[key]


def _fit_plan(idx, k):
    """(jobs, stab, n_blocks): jobs = lists of (item, slot) per job; stab[l]
    maps list positions (x, y), x <= y, to (slot, transposed) and (x, "Q") to
    the cross block's slot."""
    L_t = len(idx)
    lays = [plan_layer(idx, k, l) for l in range(L_t)]
    jobs, stab, base = [], [], []
    nu = 0
    for items, job, n_jobs in lays:
        base.append(nu)
        for j in range(n_jobs):
            jobs.append([(items[t], nu + t) for t in range(len(items)) if job[t] == j])
        nu += len(items)
    for l in range(L_t):
        s = [int(v) for v in idx[l]]
        items = lays[l][0]
        st = {}
        for x in range(k):
            st[(x, "Q")] = base[l] + items.index(("x", s[x], l))
            for y in range(x, k):
                a, b = s[x], s[y]
                l0 = next(l2 for l2 in range(L_t) if a in list(idx[l2]) and b in list(idx[l2]))
                it0 = lays[l0][0]
                if ("p", a, b) in it0:
                    st[(x, y)] = (base[l0] + it0.index(("p", a, b)), False)
                else:
                    st[(x, y)] = (base[l0] + it0.index(("p", b, a)), True)
        stab.append(st)
    return jobs, stab, nu


def decode(mode, L_s, L_t, H, k, idx, job):
    """Blocks (wave, pa, pb, out, key) of one job, as the kernel decodes them."""
    nsrc = L_s * 2 * H
    if mode == 0:
        jobs, _, nu = fit_plan(idx, k)
        hk, jj = divmod(job, len(jobs))
        kv, h = hk & 1, hk >> 1
        blocks = []
        for w, (it, slot) in enumerate(jobs[jj]):
            pa = (it[1] * 2 + kv) * H + h
            if it[0] == "x":
                pb = nsrc + (it[2] * 2 + kv) * H + h
                key = ("xy", it[2], h, kv, it[1])
            else:
                pb = (it[2] * 2 + kv) * H + h
                key = ("xx", h, kv, it[1], it[2])
            blocks.append((w, pa, pb, hk * nu + slot, key))
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


def n_jobs(mode, L_s, L_t, H, k, idx=None):
    if mode == 0:
        return H * 2 * len(fit_plan(idx, k)[0])
    return H * 2 * (((L_s + 1) // 2) * ((L_t + 1) // 2) + (L_s + 3) // 4)


def _lists(kind, L_s, L_t, k, seed):
    rng = np.random.default_rng(seed)
    if kind == "sorted":
        return np.stack([np.sort(rng.choice(L_s, k, replace=False)) for _ in range(L_t)])
    if kind == "unsorted":
        return np.stack([rng.choice(L_s, k, replace=False) for _ in range(L_t)])
    if kind == "permuted":     # one set of sources in a different order per layer
        base = rng.choice(L_s, k, replace=False)
        return np.stack([rng.permutation(base) for _ in range(L_t)])
    return np.stack([rng.choice(L_s, k, replace=True) for _ in range(L_t)])   # repeats


@pytest.mark.parametrize("k", [1, 2, 3, 4])
@pytest.mark.parametrize("shape", [(40, 64, 2), (5, 3, 2), (1, 1, 1)])
@pytest.mark.parametrize("kind", ["sorted", "unsorted", "permuted", "repeats"])
def test_fit_plan_computes_each_distinct_block_once(k, shape, kind):
    L_s, L_t, H = shape
    if k > L_s and kind != "repeats":
        pytest.skip("k > L_s")
    idx = _lists(kind, L_s, L_t, k, seed=k)
    P = (L_s + L_t) * 2 * H
    nbl = k * (k + 3) // 2
    jobs, stab, nu = fit_plan(idx, k)
    pairs = {frozenset((int(a), int(b))) for row in idx for a in row for b in row}
    cross = sum(len(set(int(v) for v in row)) for row in idx)
    assert nu == len(pairs) + cross <= L_t * nbl
    seen, outs = set(), set()
    for job in range(n_jobs(0, L_s, L_t, H, k, idx)):
        kv, blocks = decode(0, L_s, L_t, H, k, idx, job)
        assert 1 <= len(blocks) <= 4
        assert len(planes_of(blocks)) <= MAXPLANES
        for w, pa, pb, out, key in blocks:
            assert 0 <= pa < P and 0 <= pb < P
            assert kv == 1 or 0 <= P + lo_slot(H, pa) < P + P // 2
            assert 0 <= out < H * 2 * nu
            assert key not in seen and out not in outs
            seen.add(key)
            outs.add(out)
    assert outs == set(range(H * 2 * nu))
    # the solve of every task finds each block of its design and cross Gram
    slot_item = {slot: it for jb in jobs for it, slot in jb}
    for l in range(L_t):
        s = [int(v) for v in idx[l]]
        for x in range(k):
            assert slot_item[stab[l][(x, "Q")]] == ("x", s[x], l)
            for y in range(x, k):
                slot, tr = stab[l][(x, y)]
                want = ("p", s[y], s[x]) if tr else ("p", s[x], s[y])
                assert slot_item[slot] == want
                assert not (tr and s[x] == s[y])


def test_fit_plan_on_the_qwen3_14b_32b_lists():
    """The bench's index lists: 347 distinct source pairs and 256 cross blocks
    per (head, K|V) in 186 jobs, against 896 blocks in 256 jobs when every
    target layer computes all of its own."""
    from paper_2608_03893_amd import synth
    cfg = synth.CONFIGS["qwen3_14b_32b"]
    idx = synth._draw_idx(cfg, np.random.default_rng(cfg.seed))
    jobs, _, nu = fit_plan(idx, cfg.k)
    assert (nu, len(jobs)) == (603, 186)


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
    chunks = 4                                  # partial channel sums per 8192 tokens
    stride = 128 * Npad + 2176                  # token-tiled plane and its pad (elements)
    base = up(32768 * 128 * 12) + up((P + P // 2) * stride * 2) + 2 * up(chunks * P * 128 * 8)
    fit_blocks = 64 * 8 * 2 * 14
    plan = up(64 * 96) + up(64 * 14 * 32) + up(64 * 25 * 4)
    assert kvx.fit_workspace_bytes(d) == (base + up(fit_blocks * 128 * 128 * 4)
                                          + up(64 * 8 * 2 * 512 * 512 * 8)
                                          + up(64 * 8 * 2 * 512 * 128 * 8) + plan)
    assert kvx.probe_workspace_bytes(d) == base + up(40 * 8 * 2 * 65 * 128 * 128 * 4)
    assert kvx.fit_workspace_bytes(kvx.Dims(L_s=4, L_t=3, H=2, T=0, d=128, k=2)) == 0
    assert kvx.fit_workspace_bytes(kvx.Dims(L_s=4, L_t=3, H=2, T=64, d=64, k=2)) == 0
    assert kvx.fit_workspace_bytes(kvx.Dims(L_s=4, L_t=3, H=2, T=64, d=128, k=5)) == 0
