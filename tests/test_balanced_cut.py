"""CPU model of the attention kernel's balanced decomposition of dense launches, with the host
plan that bounds it, checked for the properties the kernel's buffers rely on.

The kernel (paper_2510_09883_amd/csrc/attn_kernel.hip, balanced instantiation) and the host
plan (delta_api.cpp: plan_split, plan_balance) are mirrored here step for step: the batch's
16-row groups, in (sequence, KV head, page) order, are cut into runs of
max(ceil(work / workgroups), chunk_min) groups, run w for workgroup w; the cut is taken only
when a run is at most twice the shortest pair and at most 0.9 of the static piece.  For many
random batches this checks that every page of every pair is covered exactly once, that a pair's
partial slots are exactly 0 .. n-1 and within the workspace's slots, that no piece exceeds the
1024-entry page list and that no run covers more than three pairs; equal and nearly equal
lengths keep the static plan, ragged ones get even runs.
"""
import random

KMAX_ROWS, KMAX_SPLITS, BAL_MAX_BATCH = 1024, 64, 64


def cdiv(a, b):
    return (a + b - 1) // b


def host_plan(B, Hkv, max_groups, target=256, min_gps=8, max_splits=16):
    pairs = B * Hkv
    n_split = min(max(1, cdiv(target, pairs)), max(1, cdiv(max_groups, min_gps)), max_splits)
    gps = min(cdiv(max_groups, n_split), KMAX_ROWS)
    n_split = cdiv(max_groups, gps)
    chunk_min = max(min_gps, cdiv(max_groups, min(max_splits, KMAX_SPLITS - 1)))
    balance = 2 <= B <= BAL_MAX_BATCH and chunk_min <= KMAX_ROWS and pairs * max_groups < 2 ** 31
    slots = max(n_split, cdiv(max_groups, chunk_min) + 1) if balance else n_split
    return dict(n_split=n_split, gps=gps, n_wg=n_split * pairs, chunk_min=chunk_min,
                slots=slots, balance=balance)


def pieces(lens, Hkv, max_groups, plan):
    """Per workgroup: the pieces (b, g, g0, n, slot, n_valid) it attends to."""
    B = len(lens)
    n_groups = [min(cdiv(max(s, 0), 16), max_groups) for s in lens]
    units = [max(1, n) for n in n_groups]
    before = [sum(units[:b]) for b in range(B)]
    W = Hkv * sum(units)
    chunk = max(cdiv(W, plan["n_wg"]), plan["chunk_min"])
    balanced = plan["balance"] and chunk <= 2 * min(units) and 10 * chunk <= 9 * plan["gps"]
    out = []
    for w in range(plan["n_wg"]):
        segs = []
        if balanced:
            x, xe = w * chunk, min(W, (w + 1) * chunk)
            while x < xe:
                b = sum(1 for v in before if Hkv * v <= x) - 1
                loc = x - Hkv * before[b]
                g, g0 = loc // units[b], loc % units[b]
                off = Hkv * before[b] + g * units[b]
                end = min(xe, off + units[b])
                first = off // chunk
                n_valid = (off + units[b] - 1) // chunk - first + 1
                if n_groups[b] == 0:
                    segs.append((b, g, 0, 0, 0, 0))
                else:
                    segs.append((b, g, g0, end - x, w - first, n_valid))
                x = end
        else:
            split, g = w % plan["n_split"], (w // plan["n_split"]) % Hkv
            b = w // (plan["n_split"] * Hkv)
            n_valid = cdiv(n_groups[b], plan["gps"])
            g0 = split * plan["gps"]
            if n_valid == 0 and split == 0:
                segs.append((b, g, 0, 0, 0, 0))
            elif split < n_valid:
                segs.append((b, g, g0, min(plan["gps"], n_groups[b] - g0), split, n_valid))
        out.append(segs)
    return out, balanced


def check(lens, Hkv, max_groups, **kw):
    plan = host_plan(len(lens), Hkv, max_groups, **kw)
    out, balanced = pieces(lens, Hkv, max_groups, plan)
    covered, slots = set(), {}
    for segs in out:
        assert len(segs) <= (3 if balanced else 1)
        for b, g, g0, n, slot, n_valid in segs:
            assert n <= KMAX_ROWS
            assert 0 <= slot < max(n_valid, 1) <= plan["slots"] <= KMAX_SPLITS
            slots.setdefault((b, g), []).append((slot, n_valid))
            for p in range(g0, g0 + n):
                assert (b, g, p) not in covered
                covered.add((b, g, p))
    for b, s in enumerate(lens):
        for g in range(Hkv):
            assert all((b, g, p) in covered for p in range(min(cdiv(max(s, 0), 16), max_groups)))
            got = sorted(slots[(b, g)])
            assert [x[0] for x in got] == list(range(max(got[0][1], 1)))
            assert all(x[1] == got[0][1] for x in got)
    return plan, out, balanced


def test_equal_lengths_keep_the_static_splits():
    # including page counts that are not a multiple of the static piece (65 pages in two
    # splits): a cut through the batch would drift through the pairs and leave slivers
    for lens, Hkv, mg in [([8192] * 2, 8, 512), ([32768] * 16, 8, 2048), ([32768] * 8, 4, 2048),
                          ([18432] * 64, 2, 1152), ([1024] * 3, 2, 64), ([1040] * 64, 2, 65),
                          ([1040, 1041] * 32, 2, 66), ([30000] * 24, 8, 1875)]:
        plan, out, balanced = check(lens, Hkv, mg)
        assert not balanced
        for w, segs in enumerate(out):
            split = w % plan["n_split"]
            assert segs == [] or (len(segs) == 1 and segs[0][2] == split * plan["gps"]
                                  and segs[0][4] == split)


def test_ragged_batch_is_spread_evenly():
    r = random.Random(5000)
    lens = [r.randint(16384, 32768) for _ in range(32)]
    plan, out, balanced = check(lens, 8, 2048)
    assert balanced
    loads = [sum(seg[3] for seg in segs) for segs in out]
    # every workgroup gets one run of the same length (the last one possibly shorter)
    assert max(loads) == loads[0] and max(loads) < 2048 // 2


def test_random_batches_cover_every_page_once():
    rng = random.Random(1)
    seen_balanced = 0
    for _ in range(400):
        B, Hkv, mg = rng.randint(1, 64), rng.choice([1, 2, 4, 8]), rng.randint(1, 300)
        kind = rng.random()
        if kind < 0.3:
            lens = [rng.randint(1, 16 * mg) for _ in range(B)]
        elif kind < 0.6:
            lens = [rng.randint(8 * mg, 16 * mg) for _ in range(B)]
        elif kind < 0.8:
            lens = [16 * mg] * B
        else:
            lens = [rng.choice([0, 1, 16 * mg, rng.randint(1, 16 * mg)]) for _ in range(B)]
        _, _, balanced = check(lens, Hkv, mg, target=rng.choice([256, 512, 64]))
        seen_balanced += balanced
    assert seen_balanced > 80


def test_gpu_test_batches_take_the_balanced_cut():
    """Every batch of tests/test_gpu_balanced.py that is meant to run the balanced cut takes it
    under the model above (and the batch one past the lane limit does not), so a change to the
    cut's threshold cannot move those GPU tests onto the static split unnoticed."""
    import balanced_cases as BC
    for _, hkv, lens in BC.RAGGED:
        assert check(lens, hkv, cdiv(max(lens), 16))[2], lens
    for _, seed in BC.RANDOM:
        hkv, _, lens = BC.random_case(seed)
        assert check(lens, hkv, cdiv(max(lens), 16))[2], seed
    for B in BC.BATCH_LIMIT:
        lens = BC.batch_limit_lens(B)
        taken = check(lens, BC.BATCH_LIMIT_KV_HEADS, cdiv(max(lens), 16))[2]
        assert taken == (B <= BAL_MAX_BATCH), B
