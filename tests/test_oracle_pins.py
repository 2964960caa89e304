"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: a hand trace
(tests/golden), a closed form, a brute-force set computation, or an invariant
the paper states.  None of them calls the GPU path.
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def life_of(q):
    return ((np.asarray(q, dtype=np.uint32) >> 24).astype(np.uint8)).astype(np.int8).astype(np.int32)


# ---------------------------------------------------------------------------
# metadata word (Eq. 2, Eq. 3, Appendix F)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("m", [1, 3, 10, 13, 16, 22, 23])
def test_word_layout_matches_eq2(oracle_lib, m):
    """Fields from MSB to LSB: lifetime 8 | invalid 1 | fingerprint 23-m | slot m."""
    S, F = 1 << m, 1 << (23 - m)
    assert O.pack(m, 0, 0, 0, 1) == 1
    assert O.pack(m, 0, 0, 0, S - 1) == S - 1
    if F > 1:
        assert O.pack(m, 0, 0, 1, 0) == 1 << m
        assert O.pack(m, 0, 0, F - 1, 0) == (F - 1) << m
    assert O.pack(m, 0, 1, 0, 0) == 1 << 23
    assert O.pack(m, 1, 0, 0, 0) == 1 << 24
    assert O.pack(m, 127, 0, 0, 0) == 127 << 24
    # two's-complement lifetime byte: -1 fills the top byte
    assert O.pack(m, -1, 0, 0, 0) == 0xFF000000
    assert O.pack(m, -1, 1, F - 1, S - 1) == 0xFFFFFFFF


@pytest.mark.parametrize("m", [3, 10, 13, 23])
def test_decode_chain_inverts_pack(oracle_lib, m):
    """Appendix F decode of an Eq. 3 word returns the packed fields."""
    S, F = 1 << m, 1 << (23 - m)
    rng = np.random.default_rng(m)
    for _ in range(300):
        l = int(rng.integers(-1, 128))
        b = int(rng.integers(0, 2))
        fp = int(rng.integers(0, F))
        o = int(rng.integers(0, S))
        assert O.decode(m, O.pack(m, l, b, fp, o)) == (l, b, fp, o)


def test_fingerprint_of_empty_id(oracle_lib):
    """phi(x) = x mod F taken non-negative: phi(-1) = F - 1; phi(x + F) = phi(x)."""
    for m in (3, 13):
        F = 1 << (23 - m)
        assert O.phi(m, -1) == F - 1
        assert O.phi(m, 5) == 5 % F
        assert O.phi(m, 5 + F) == O.phi(m, 5)


# ---------------------------------------------------------------------------
# hand trace
# ---------------------------------------------------------------------------
def test_hand_trace_s8(oracle_lib):
    g = json.load(open(os.path.join(GOLDEN, "hand_trace_s8.json")))
    c = g["config"]
    orc = O.Oracle(c["batch"], c["topk"], c["n_q"], c["slots"], c["retry"], c["max_life"],
                   c["a1"], c["a2"], nthreads=1)
    for k, s in enumerate(g["steps"]):
        X = np.array(s["X"], dtype=np.int32)[None]
        Ot, n = orc.step(X, np.array([s["N"]], dtype=np.int64))
        assert Ot[0].tolist() == s["O"], f"step {k}"
        assert n[0].tolist() == s["n"], f"step {k}"
        mx, mo = orc.misses(0, n[0])
        assert mx.tolist() == s["miss_x"] and mo.tolist() == s["miss_o"], f"step {k}"
    cc, q = orc.export(0)
    assert cc.tolist() == g["final_c"]
    assert life_of(q).tolist() == g["final_life"]
    for j, (b, fp, slot) in enumerate(g["final_buckets"]):
        l, bb, ff, oo = O.decode(3, int(q[j]))
        assert (bb, ff, oo) == (b, fp, slot), f"bucket {j}"
    assert {k: v for k, v in orc.stats(0).items() if k in g["counters"]} == g["counters"]


# ---------------------------------------------------------------------------
# closed forms
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("S,seed", [(8, 0), (16, 1), (64, 2)])
def test_no_eviction_closed_form(oracle_lib, S, seed):
    """K = 1, N_q = 1, R = S - 1, L >= T, at most S distinct ids: no slot ever
    dies and every install finds a reusable bucket, so a lookup hits exactly
    when its id was seen before, and an id's slot is the rank of its first
    appearance."""
    rng = np.random.default_rng(seed)
    T = 60
    universe = rng.choice(10_000_000, size=S, replace=False)
    ids = universe[rng.integers(0, S, size=T)]
    orc = O.Oracle(1, 1, 1, S, retry=S - 1, max_life=T + 1, nthreads=1)
    first_rank = {}
    for t, x in enumerate(ids):
        Ot, n = orc.step(np.array([[[x]]], dtype=np.int32))
        seen = x in first_rank
        if not seen:
            first_rank[x] = len(first_rank)
        assert n[0, 0] == (0 if seen else 1), t
        assert Ot[0, 0, 0] == first_rank[x], t
    st_ = orc.stats(0)
    assert st_["lost_exhausted"] == 0 and st_["alloc_decays"] == 0


@pytest.mark.parametrize("S,L", [(4, 2), (8, 3), (16, 1), (16, 15)])
def test_lifetime_aging_closed_form(oracle_lib, S, L):
    """K = 1, a fresh id every step: a slot set to L becomes reclaimable after
    L + 1 unrefreshed steps and dead slots are taken in increasing order, so
    step t uses slot t mod (L + 1) (needs S >= L + 1)."""
    orc = O.Oracle(1, 1, 1, S, retry=3, max_life=L, nthreads=1)
    for t in range(4 * (L + 1) + 3):
        Ot, n = orc.step(np.array([[[1000 + t]]], dtype=np.int32))
        assert n[0, 0] == 1
        assert Ot[0, 0, 0] == t % (L + 1), t
    # a slot whose lifetime is zero is not reclaimable: lifetimes after the last step
    c, q = orc.export(0)
    lives = sorted(life_of(q)[: L + 1].tolist())
    assert lives == list(range(0, L + 1))


def test_refresh_keeps_an_id_resident(oracle_lib):
    """An id selected every step is refreshed to L on each hit and never evicted,
    while ids selected once expire; with R = S - 1 nothing is lost."""
    S, L, K = 16, 2, 2
    orc = O.Oracle(1, K, 1, S, retry=S - 1, max_life=L, nthreads=1)
    slot_a = None
    for t in range(40):
        X = np.array([[[7, 100 + t]]], dtype=np.int32)
        Ot, n = orc.step(X)
        if t == 0:
            assert n[0, 0] == 2
            slot_a = Ot[0, 0, 0]
        else:
            assert Ot[0, 0, 0] == slot_a
            assert n[0, 0] == 1


# ---------------------------------------------------------------------------
# brute force on tiny inputs
# ---------------------------------------------------------------------------
def _brute_force_run(S, K, R, L, U, T, seed, exact_required=False):
    rng = np.random.default_rng(seed)
    orc = O.Oracle(1, K, 1, S, retry=R, max_life=L, nthreads=1)
    exact_steps = 0
    for t in range(T):
        c_before, q_before = orc.export(0)
        life_after_decay = np.maximum(life_of(q_before) - 1, -1)
        X = rng.choice(U, size=K, replace=False).astype(np.int32)
        before = orc.stats(0)
        Ot, n = orc.step(X[None, None])
        after = orc.stats(0)
        hit_count = K - n[0, 0]
        resident = set(c_before.tolist())
        o = Ot[0, 0]
        # the transfer list names the misses (ids are distinct within a token)
        mx, mo = orc.misses(0, n[0])
        assert mx.tolist() == [int(x) for x in X if int(x) in set(mx.tolist())]
        hit = ~np.isin(X, mx)
        assert hit.sum() == hit_count
        for i in range(K):
            if hit[i]:
                # soundness: a hit names a slot that held the id before the step
                assert X[i] in resident and c_before[o[i]] == X[i]
        # o is a function from slots to ids within the step
        assert len(set(o.tolist())) == K
        # no install lost before this step: every id held by an active slot hits
        if before["lost_exhausted"] == 0 and before["lost_collision"] == 0:
            active = {int(c_before[j]) for j in range(S) if life_after_decay[j] >= 0 and c_before[j] >= 0}
            must_hit = np.array([int(x) in active for x in X])
            assert np.all(hit[must_hit]), (t, X, c_before, life_after_decay)
            # and with no revival either, the hits are exactly x ∩ active
            if after["revivals"] == 0:
                assert np.array_equal(hit, must_hit)
            exact_steps += 1
    if exact_required:
        assert exact_steps == T
    return exact_steps


@settings(max_examples=60, deadline=None)
@given(st.sampled_from([8, 16, 32, 64]), st.integers(1, 8), st.integers(0, 4),
       st.integers(1, 6), st.integers(1, 4), st.integers(0, 2**31 - 1))
def test_brute_force_intersection(oracle_lib, S, K_, R, L, u_mul, seed):
    """Hits are always a subset of x ∩ {c_j}; while no install has been lost and
    no dead slot revived, hits equal x ∩ {c_j : lifetime_j >= 0 after the
    step's pre-decay}, because a live mapping to an active slot is never
    reusable and so survives until the slot dies (Eq. 4)."""
    K = min(K_, S)
    U = max(K, (S * u_mul) // 2)
    _brute_force_run(S, K, min(R, S - 1), L, U, 12, seed)


def test_brute_force_exact_regime(oracle_lib):
    """R = S - 1 and K = 1: no install is ever lost, so every step is checked
    against the set bounds x ∩ active <= hits <= x ∩ resident."""
    for seed in range(5):
        _brute_force_run(16, 1, 15, 3, 24, 50, seed, exact_required=True)


# ---------------------------------------------------------------------------
# invariants on seeded workloads, with Stage Two into a host image
# ---------------------------------------------------------------------------
def _make_rows(B, rows, rb, rng):
    return [np.ascontiguousarray(rng.integers(0, 256, size=(rows, rb), dtype=np.uint8)) for _ in range(B)]


@pytest.mark.parametrize("B,K,n_q,S,L,R,U,T", [
    (3, 16, 1, 32, 4, 3, 80, 30),
    (2, 16, 2, 32, 4, 3, 60, 30),
    (2, 8, 3, 32, 2, 1, 40, 30),
    (2, 32, 4, 128, 16, 3, 300, 20),
])
def test_invariants(oracle_lib, B, K, n_q, S, L, R, U, T):
    """hits + misses = K per token; no slot holds two ids within a request-step;
    allocation decays per request-step stay within L when S >= N_q*K; every
    selected index's slot holds exactly its host row after Stage Two."""
    rng = np.random.default_rng(B * 1000 + K)
    rb = 24
    host = _make_rows(B, U, rb, rng)
    buf = [np.zeros((S, rb), dtype=np.uint8) for _ in range(B)]
    orc = O.Oracle(B, K, n_q, S, retry=R, max_life=L, nthreads=2)
    for t in range(T):
        X = np.stack([np.stack([rng.choice(U, size=K, replace=False) for _ in range(n_q)])
                      for _ in range(B)]).astype(np.int32)
        Ot, n = orc.step(X, host=[h.ctypes.data for h in host], buf=[b.ctypes.data for b in buf],
                         row_bytes=[rb])
        for r in range(B):
            slot_to_id = {}
            for g in range(n_q):
                assert 0 <= n[r, g] <= K
                for i in range(K):
                    o = int(Ot[r, g, i])
                    assert 0 <= o < S
                    assert slot_to_id.setdefault(o, int(X[r, g, i])) == X[r, g, i]
                    assert np.array_equal(buf[r][o], host[r][X[r, g, i]])
            mx, mo = orc.misses(r, n[r])
            assert len(set(mo.tolist())) == len(mo)   # a slot is reserved once per step
    assert orc.total_stats()["max_step_alloc_decays"] <= L


def test_mtp_cold_start(oracle_lib):
    """From an empty table the first token has no hits (every slot is empty),
    and a later token repeating the first token's selection hits every id whose
    reservation was installed (shared buffer across MTP tokens)."""
    K, S = 64, 256
    rng = np.random.default_rng(3)
    orc = O.Oracle(1, K, 2, S, retry=3, max_life=16, nthreads=1)
    x = rng.choice(100000, size=K, replace=False)
    X = np.stack([x, rng.permutation(x)])[None].astype(np.int32)
    Ot, n = orc.step(X)
    st_ = orc.stats(0)
    lost = st_["lost_exhausted"] + st_["lost_collision"]
    assert n[0, 0] == K
    assert n[0, 1] == lost
    # a later token's hits use the same slots as the first token's reservations
    slot_of = dict(zip(X[0, 0].tolist(), Ot[0, 0].tolist()))
    mx, mo = orc.misses(0, n[0])
    missed_twice = set(mx[K:].tolist())
    for i, xi in enumerate(X[0, 1].tolist()):
        if xi not in missed_twice:
            assert Ot[0, 1, i] == slot_of[xi]


def test_speculative_invalidation(oracle_lib):
    """Ids >= N are cleared at the end of the step, so a later selection of the
    same position misses and refetches the regenerated host row."""
    B, K, n_q, S, rb = 1, 8, 2, 32, 16
    rng = np.random.default_rng(5)
    U = 64
    host = _make_rows(B, U, rb, rng)
    buf = [np.zeros((S, rb), dtype=np.uint8)]
    N = 40
    orc = O.Oracle(B, K, n_q, S, nthreads=1)
    X = np.array([[[41, 42, 1, 2, 3, 4, 5, 6], [41, 42, 1, 2, 3, 4, 5, 7]]], dtype=np.int32)
    orc.step(X, np.array([N]), host=[host[0].ctypes.data], buf=[buf[0].ctypes.data], row_bytes=[rb])
    c, _ = orc.export(0)
    assert not np.any(c >= N)
    assert orc.stats(0)["invalidations"] == 2
    host[0][41] ^= 0xFF   # the speculative rows are regenerated
    host[0][42] ^= 0xFF
    Ot, n = orc.step(X, np.array([N]), host=[host[0].ctypes.data], buf=[buf[0].ctypes.data],
                     row_bytes=[rb])
    for g in range(2):
        for i in range(K):
            assert np.array_equal(buf[0][Ot[0, g, i]], host[0][X[0, g, i]])
    mx, _ = orc.misses(0, n[0])
    assert {41, 42} <= set(mx.tolist())


def test_missing_invalidation_is_caught(oracle_lib):
    """Mutation check on the CPU: without the end-of-step invalidation the
    regenerated speculative rows would be served stale, and the content
    invariant used by the parity tests detects it."""
    B, K, n_q, S, rb = 1, 8, 2, 32, 16
    rng = np.random.default_rng(5)
    host = _make_rows(B, 64, rb, rng)
    buf = [np.zeros((S, rb), dtype=np.uint8)]
    orc = O.Oracle(B, K, n_q, S, nthreads=1)
    X = np.array([[[41, 42, 1, 2, 3, 4, 5, 6], [41, 42, 1, 2, 3, 4, 5, 7]]], dtype=np.int32)
    kw = dict(host=[host[0].ctypes.data], buf=[buf[0].ctypes.data], row_bytes=[rb])
    orc.step(X, None, **kw)     # no verified length: no invalidation
    host[0][41] ^= 0xFF
    Ot, n = orc.step(X, None, **kw)
    stale = [not np.array_equal(buf[0][Ot[0, 0, i]], host[0][X[0, 0, i]]) for i in range(K)]
    assert any(stale)


def test_slot_preservation_bound(oracle_lib):
    """With S = N_q*K exactly and every index distinct, the cumulative
    allocation decays of a request-step never exceed L, and no slot output
    earlier in the step is reclaimed (Appendix B, slot preservation)."""
    K, n_q, L = 16, 4, 3
    S = K * n_q
    rng = np.random.default_rng(9)
    orc = O.Oracle(2, K, n_q, S, retry=2, max_life=L, nthreads=1)
    for t in range(40):
        X = rng.choice(10**6, size=(2, n_q * K), replace=False).reshape(2, n_q, K).astype(np.int32)
        Ot, n = orc.step(X)
        for r in range(2):
            assert len(set(Ot[r].ravel().tolist())) == n_q * K
    assert orc.total_stats()["max_step_alloc_decays"] <= L


# ---------------------------------------------------------------------------
# Probe chains (Eq. 8-11)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("S", [8, 64])
def test_probe_chain_covers_all_buckets(oracle_lib, S):
    """Strides are odd and S is a power of two, so with R = S - 1 the chain of
    any id visits every bucket: a mapping placed in any bucket is found.  With
    R = 0 exactly one bucket is examined."""
    m = S.bit_length() - 1
    orc_full = O.Oracle(1, 1, 1, S, retry=S - 1, nthreads=1)
    orc_one = O.Oracle(1, 1, 1, S, retry=0, nthreads=1)
    x, slot = 123457, 5
    c = np.full(S, -1, dtype=np.int32)
    c[slot] = x
    inv = O.pack(m, 0, 1, 0, 0)
    found_once = []
    for b in range(S):
        q = np.full(S, inv, dtype=np.uint32)
        q[b] = O.pack(m, 0, 0, O.phi(m, x), slot)
        orc_full.import_table(0, c, q)
        orc_one.import_table(0, c, q)
        hit, h = orc_full.probe(0, x)
        assert hit and h == b
        hit1, _ = orc_one.probe(0, x)
        found_once.append(hit1)
    assert sum(found_once) == 1


def test_probe_ignores_invalid_flag_and_lifetime(oracle_lib):
    """A hit only needs the full id comparison: an invalid bucket or a dead
    slot still yields a hit when the pointed slot holds the id."""
    S, m = 8, 3
    x = 11
    orc = O.Oracle(1, 1, 1, S, retry=S - 1, nthreads=1)
    c = np.full(S, -1, dtype=np.int32)
    c[2] = x
    q = np.full(S, O.pack(m, -1, 1, 0, 2), dtype=np.uint32)  # every bucket: invalid, slot 2
    orc.import_table(0, c, q)
    hit, _ = orc.probe(0, x)
    assert hit
    hit2, _ = orc.probe(0, x + 1)
    assert not hit2


# ---------------------------------------------------------------------------
# dual-pointer baseline
# ---------------------------------------------------------------------------
def test_dual_pointer_exact(oracle_lib):
    """Sort-merge matching with S = K: hits are exactly x_t ∩ x_{t-1}, hit slots
    keep their position, and after the step the buffer holds x_t."""
    B, K, U = 3, 64, 200
    rng = np.random.default_rng(11)
    dp = O.DualPointerOracle(B, K, nthreads=2)
    prev = [None] * B
    prev_slot = [None] * B
    for t in range(25):
        X = np.stack([rng.choice(U, size=K, replace=False) for _ in range(B)]).astype(np.int32)
        Ot, n = dp.step(X)
        for r in range(B):
            x = X[r].tolist()
            o = Ot[r, 0].tolist()
            inter = set(x) & set(prev[r] or [])
            assert K - n[r, 0] == len(inter)
            assert sorted(o) == list(range(K))
            cached = dp.export(r)
            assert set(cached.tolist()) == set(x)
            for i, xi in enumerate(x):
                assert cached[o[i]] == xi
                if xi in inter:
                    assert o[i] == prev_slot[r][xi]
            prev[r] = x
            prev_slot[r] = dict(zip(x, o))


# ---------------------------------------------------------------------------
# Stage Two assignments (Appendix D)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("N,C", [(0, 7), (5, 7), (1000, 256), (19203, 1024), (262144, 1024)])
def test_balanced_partition(oracle_lib, N, C):
    """Eq. 6: consecutive ranges covering every miss once, sizes floor/ceil of N/C."""
    b = O.partition_balanced(N, C)
    assert b[0] == 0 and b[-1] == N
    sizes = np.diff(b)
    assert np.all(sizes >= 0)
    assert set(sizes.tolist()) <= {N // C, -(-N // C)}
    assert sizes.max() - sizes.min() <= 1


@pytest.mark.parametrize("B,C", [(1, 256), (64, 256), (300, 256), (512, 256)])
def test_request_partition(oracle_lib, B, C):
    """Eq. 13: the first B mod C workers take one extra request of N_q*K positions."""
    n_q, K = 2, 2048
    p = O.partition_request(B, C, n_q, K)
    assert p.sum() == B * n_q * K
    rB = B % C
    assert np.all(p[:rB] == (B // C + 1) * n_q * K)
    assert np.all(p[rB:] == (B // C) * n_q * K)


def test_position_partition(oracle_lib):
    """Eq. 14: near-equal contiguous ranges of the N_g*K flattened positions."""
    b = O.partition_position(64 * 2 * 2048, 1000)
    s = np.diff(b)
    assert b[-1] == 64 * 2 * 2048 and s.max() - s.min() <= 1


# ---------------------------------------------------------------------------
# configuration errors
# ---------------------------------------------------------------------------
def test_config_errors(oracle_lib):
    ok = dict(batch=1, topk=4, n_q=2, slots=8)
    assert O.Oracle.create_status(**ok) == 0
    assert O.Oracle.create_status(batch=0, topk=4, n_q=1, slots=8) == -1
    assert O.Oracle.create_status(batch=1, topk=4, n_q=1, slots=12) == -2
    assert O.Oracle.create_status(batch=1, topk=8, n_q=2, slots=8) == -3   # Eq. 7
    assert O.Oracle.create_status(**ok, max_life=0) == -4
    assert O.Oracle.create_status(**ok, max_life=128) == -4
    assert O.Oracle.create_status(**ok, a1=7, a2=7) == -4
    assert O.Oracle.create_status(**ok, a1=9, a2=7) == -4   # not prime
    assert O.Oracle.create_status(**ok, retry=-1) == -4


# ---------------------------------------------------------------------------
# selection check of the validate mode (the input of Section 3.2: each token's
# top-K list holds K distinct positions of its request's context)
# ---------------------------------------------------------------------------
def test_validate_hand_cases(oracle_lib):
    """Rows checked by eye: distinct in-range ids are valid; an id below 0 or
    at or above the request's rows sets bit 0; an in-range id seen twice sets
    bit 1; an out-of-range id seen twice is only out of range."""
    X = np.array([[[0, 1, 2, 4]], [[3, 1, 3, 0]], [[-1, 1, 2, 0]], [[5, 1, 2, 0]],
                  [[7, 7, 1, 1]], [[9, 9, 0, 1]], [[4, 3, 2, 1]]], dtype=np.int32)
    rows = np.array([5, 5, 5, 5, 5, 5, 4])
    assert O.validate(X, rows).ravel().tolist() == [0, 2, 1, 1, 3, 1, 1]


def test_validate_two_tokens_share_ids(oracle_lib):
    """Tokens of one step may share indices (that is the MTP reuse of Section
    3.6); only a repeat inside one token's list is flagged, and each row is
    checked against its own request's rows."""
    X = np.array([[[0, 1, 2], [2, 1, 0]], [[6, 7, 8], [6, 6, 1]]], dtype=np.int32)
    assert O.validate(X, [3, 9]).tolist() == [[0, 0], [0, 2]]
    assert O.validate(X, [3, 8]).tolist() == [[0, 0], [1, 2]]


# ---------------------------------------------------------------------------
# resident-reuse transfer plan (a property of the transfer: every slot must end
# up with the bytes the paper's Stage Two writes)
# ---------------------------------------------------------------------------
def _replay_plan(buf, plan, rows):
    """Apply a plan to a buffer of row ids in the kernels' order: host entries
    into their slot and fan slots (ids outside [0, rows) are skipped, as by the
    copy) and resident copies, then repeat copies."""
    hx, ho, hf, rs, rd, ps, pd = plan
    res = buf[rs].copy()                    # resident sources are not written this step
    for x, o, fs in zip(hx.tolist(), ho.tolist(), hf.tolist()):
        if 0 <= x < rows:
            buf[o] = x
            for f in fs:
                if f >= 0:
                    buf[f] = x
    for v, o in zip(res.tolist(), rd.tolist()):
        buf[o] = v
    rep = buf[ps].copy()
    for v, o in zip(rep.tolist(), pd.tolist()):
        buf[o] = v


@pytest.mark.parametrize("K,n_q,S,R,L,U,T,bad", [
    (16, 2, 32, 0, 4, 60, 40, False),
    (8, 3, 32, 1, 2, 40, 40, False),
    (16, 4, 64, 0, 16, 120, 30, False),
    (16, 2, 32, 0, 4, 60, 30, True),
    (16, 6, 128, 0, 16, 200, 30, False),
])
def test_transfer_plan_replays_stage_two(oracle_lib, K, n_q, S, R, L, U, T, bad):
    """Replaying the plan on a buffer of row ids gives, step after step, the
    buffer of the paper's Stage Two (every miss copied from the host in list
    order), and device copies actually occur (R = 0 loses many installs)."""
    rng = np.random.default_rng(K * 100 + n_q)
    B = 2
    rows = U
    orc = O.Oracle(B, K, n_q, S, retry=R, max_life=L, nthreads=1)
    paper = [np.full(S, -1, dtype=np.int64) for _ in range(B)]
    plan_buf = [np.full(S, -1, dtype=np.int64) for _ in range(B)]
    n_res = n_dup = n_left = 0
    for t in range(T):
        X = np.stack([np.stack([rng.choice(U, size=K, replace=False) for _ in range(n_q)])
                      for _ in range(B)]).astype(np.int32)
        if bad:
            X[0, 0, 0] = U + 5               # outside [0, rows): never copied
        _, n = orc.step(X)                   # no index validation: a bad id takes a slot
        for r in range(B):
            mx, mo = orc.misses(r, n[r])
            for x, o in zip(mx.tolist(), mo.tolist()):
                if 0 <= x < rows:
                    paper[r][o] = x
            c, _ = orc.export(r)
            plan = O.transfer_plan(mx, mo, c, rows)
            hx, ho, hf, rs, rd, ps, pd = plan
            fanned = int(np.sum(hf >= 0))
            nr, nd = len(rs), len(ps) + fanned
            assert len(hx) + nr + nd == len(mx)
            assert not set(rs.tolist()) & set(mo.tolist())     # resident sources are not reserved
            assert set(ps.tolist()) <= set(ho.tolist())        # repeat sources get a host copy
            assert set(hf[hf >= 0].tolist()) <= set(mo.tolist()) - set(ho.tolist())
            # host entries read distinct valid rows
            valid = [x for x in hx.tolist() if 0 <= x < rows]
            assert len(valid) == len(set(valid))
            _replay_plan(plan_buf[r], plan, rows)
            assert np.array_equal(plan_buf[r], paper[r]), f"step {t} request {r}"
            n_res += nr
            n_dup += nd
            n_left += len(ps)
    assert n_res > 0 and (n_q == 1 or n_dup > 0)
    if n_q > 3:
        assert n_left > 0                    # an index missed by four tokens leaves a repeat
    else:
        assert n_left == 0                   # two fan slots cover every repeat of three tokens


def test_transfer_plan_finds_an_orphaned_slot(oracle_lib):
    """Hand case: slot 5 caches id 42 but no bucket maps to it (every bucket is
    invalid), so 42 misses, takes a dead slot, and the plan fills that slot from
    slot 5 instead of the host."""
    S, m = 8, 3
    orc = O.Oracle(1, 1, 1, S, retry=S - 1, max_life=4, nthreads=1)
    c = np.full(S, -1, dtype=np.int32)
    c[5] = 42
    q = np.full(S, O.pack(m, -1, 1, 0, 0), dtype=np.uint32)   # all buckets invalid, lifetimes -1
    q[5] = O.pack(m, 3, 1, 0, 0)                              # slot 5 alive (lifetime 3)
    orc.import_table(0, c, q)
    O_t, n = orc.step(np.array([[[42]]], dtype=np.int32), rows=np.array([100], dtype=np.int64))
    assert n[0, 0] == 1
    mx, mo = orc.misses(0, n[0])
    new = int(mo[0])
    assert new != 5
    cc, _ = orc.export(0)
    hx, ho, hf, rs, rd, ps, pd = O.transfer_plan(mx, mo, cc, 100)
    assert len(hx) == 0 and rs.tolist() == [5] and rd.tolist() == [new] and len(ps) == 0
    # with the orphan invalidated (c = -1) the row must come from the host
    cc2 = cc.copy()
    cc2[5] = -1
    hx, ho, hf, rs, rd, ps, pd = O.transfer_plan(mx, mo, cc2, 100)
    assert hx.tolist() == [42] and ho.tolist() == [new] and hf.tolist() == [[-1, -1]]
    assert len(rs) == 0 and len(ps) == 0


def test_transfer_plan_same_step_repeat(oracle_lib):
    """Hand case: the same id listed by two tokens of one step (its first
    install lost) is copied from the host once, into the larger slot, and the
    same copy writes the other slot (its first fan slot)."""
    mx = np.array([7, 9, 7], dtype=np.int32)
    mo = np.array([2, 3, 6], dtype=np.int32)
    c = np.full(8, -1, dtype=np.int32)
    c[2], c[3], c[6] = 7, 9, 7
    hx, ho, hf, rs, rd, ps, pd = O.transfer_plan(mx, mo, c, 10)
    assert hx.tolist() == [9, 7] and ho.tolist() == [3, 6] and hf.tolist() == [[-1, -1], [2, -1]]
    assert len(ps) == 0 and len(rs) == 0


def test_transfer_plan_three_tokens_repeat(oracle_lib):
    """Hand case: an id listed by three tokens: one host copy into the largest
    slot that also writes the two other slots (its fan slots, larger first)."""
    mx = np.array([7, 7, 7], dtype=np.int32)
    mo = np.array([4, 1, 3], dtype=np.int32)
    c = np.full(8, -1, dtype=np.int32)
    c[1], c[3], c[4] = 7, 7, 7
    hx, ho, hf, rs, rd, ps, pd = O.transfer_plan(mx, mo, c, 10)
    assert hx.tolist() == [7] and ho.tolist() == [4] and hf.tolist() == [[3, 1]]
    assert len(ps) == 0 and len(rs) == 0


def test_transfer_plan_four_tokens_repeat(oracle_lib):
    """Hand case: an id listed by four tokens: one host copy into the largest
    slot and its two fan slots, the smallest slot copied after from the host
    copy's slot."""
    mx = np.array([7, 7, 7, 7], dtype=np.int32)
    mo = np.array([4, 1, 6, 3], dtype=np.int32)
    c = np.full(8, -1, dtype=np.int32)
    c[1], c[3], c[4], c[6] = 7, 7, 7, 7
    hx, ho, hf, rs, rd, ps, pd = O.transfer_plan(mx, mo, c, 10)
    assert hx.tolist() == [7] and ho.tolist() == [6] and hf.tolist() == [[4, 3]]
    assert ps.tolist() == [6] and pd.tolist() == [1] and len(rs) == 0


# ---------------------------------------------------------------------------
# early-fetch transfer: rows of indices no slot held when the step began are
# read from the host before Stage One; the rest is planned as above
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("K,n_q,S,R,L,U,T,bad,share", [
    (16, 2, 32, 0, 4, 60, 40, False, 0.0),
    (8, 3, 32, 1, 2, 40, 40, False, 0.5),
    (16, 4, 64, 0, 16, 120, 30, False, 0.7),
    (16, 2, 32, 0, 4, 60, 30, True, 0.5),
    (6, 5, 32, 0, 3, 30, 30, False, 0.9),    # ids listed by all five tokens exceed four positions
])
def test_early_fetch_replays_stage_two(oracle_lib, K, n_q, S, R, L, U, T, bad, share):
    """Writing every early key's row into the slot of each of its positions and
    then replaying the plan of the remaining misses gives, step after step,
    the buffer of the paper's Stage Two.  Early keys are host entries of the
    full plan, and their positions' slots are slots the step reserved for
    them."""
    rng = np.random.default_rng(K * 1000 + n_q * 10 + int(bad))
    B = 2
    rows = U
    orc = O.Oracle(B, K, n_q, S, retry=R, max_life=L, nthreads=1)
    paper = [np.full(S, -1, dtype=np.int64) for _ in range(B)]
    early_buf = [np.full(S, -1, dtype=np.int64) for _ in range(B)]
    n_early = n_left = n_capped = 0
    for t in range(T):
        X = np.empty((B, n_q, K), dtype=np.int32)
        for r in range(B):
            X[r, 0] = rng.choice(U, size=K, replace=False)
            for g in range(1, n_q):
                x = rng.choice(U, size=K, replace=False)
                keep = rng.random(K) < share
                x[keep] = X[r, 0][keep]             # later tokens repeat some of token 0's ids
                _, first = np.unique(x, return_index=True)
                if len(first) < K:                  # keep the token's ids distinct
                    pool = np.setdiff1d(np.arange(U), x)
                    dup = np.setdiff1d(np.arange(K), first)
                    x[dup] = rng.choice(pool, size=len(dup), replace=False)
                X[r, g] = x
        if bad:
            X[0, 0, 0] = U + 5
        before = [orc.export(r)[0] for r in range(B)]
        O_t, n = orc.step(X)
        for r in range(B):
            mx, mo = orc.misses(r, n[r])
            for x, o in zip(mx.tolist(), mo.tolist()):
                if 0 <= x < rows:
                    paper[r][o] = x
            keys, where = O.early_set(X[r], before[r], rows)
            counts = {}
            for x in X[r].ravel().tolist():
                counts[x] = counts.get(x, 0) + 1
            n_capped += sum(1 for x, c in counts.items()
                            if 0 <= x < rows and c > O.EARLY_MAX_POSITIONS and x not in before[r])
            c_after, _ = orc.export(r)
            full = O.transfer_plan(mx, mo, c_after, rows)
            host_keys = {int(x) for x in full[0].tolist() if 0 <= x < rows}
            assert set(keys.tolist()) <= host_keys
            flat = O_t[r].ravel()
            for x, ps in zip(keys.tolist(), where):
                reserved = {int(o) for xx, o in zip(mx.tolist(), mo.tolist()) if xx == x}
                assert {int(flat[p]) for p in ps} == reserved
                for p in ps:
                    early_buf[r][flat[p]] = x
            rest = O.transfer_plan_early(mx, mo, c_after, rows, keys)
            _replay_plan(early_buf[r], rest, rows)
            assert np.array_equal(early_buf[r], paper[r]), f"step {t} request {r}"
            n_early += len(keys)
            n_left += len([x for x in rest[0].tolist() if 0 <= x < rows])
    assert n_early > 0
    if n_q == 5:
        assert n_capped > 0


def test_early_set_excludes_cached_indices(oracle_lib):
    """Hand case: id 42 sits in dead slot 0 with no bucket mapping it, id 43 is
    nowhere.  Both miss; 42 takes slot 0 (the first dead slot), which already
    holds its row, and 43 takes slot 1.  Only 43 is an early key; 42, cached
    when the step began, stays with the planned transfer as a host entry (its
    only copy is in a slot this step reserved)."""
    S, m = 8, 3
    orc = O.Oracle(1, 2, 1, S, retry=S - 1, max_life=4, nthreads=1)
    c = np.full(S, -1, dtype=np.int32)
    c[0] = 42
    q = np.full(S, O.pack(m, -1, 1, 0, 3), dtype=np.uint32)   # every bucket names empty slot 3
    orc.import_table(0, c, q)
    before = orc.export(0)[0]
    X = np.array([[[42, 43]]], dtype=np.int32)
    O_t, n = orc.step(X, rows=np.array([100], dtype=np.int64))
    assert n[0, 0] == 2 and O_t[0, 0].tolist() == [0, 1]
    keys, where = O.early_set(X[0], before, 100)
    assert keys.tolist() == [43] and where == [[1]]
    mx, mo = orc.misses(0, n[0])
    c_after, _ = orc.export(0)
    hx, ho, hf, rs, rd, ps, pd = O.transfer_plan_early(mx, mo, c_after, 100, keys)
    assert hx.tolist() == [42] and ho.tolist() == [0] and len(rs) == 0 and len(ps) == 0
    full = O.transfer_plan(mx, mo, c_after, 100)
    assert full[0].tolist() == [42, 43]


def test_early_set_positions_and_limits(oracle_lib):
    """Hand case: positions are flat g * K + i; an id at five positions (beyond
    four), an out-of-range id and a cached id are not early keys."""
    X = np.array([[5, 9, 2], [9, 5, 3], [9, 4, 7], [9, 8, 6], [9, 1, 0]], dtype=np.int32)
    c = np.array([-1, 3, -1, -1], dtype=np.int32)
    keys, where = O.early_set(X, c, rows_r=9)
    assert keys.tolist() == [0, 1, 2, 4, 5, 6, 7, 8]
    assert where[keys.tolist().index(5)] == [0, 4]
    assert 9 not in keys.tolist() and 3 not in keys.tolist()
