"""Pins of the CPU oracle to what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every check is a closed form, a
value the paper prints (tests/golden/, each with its citation), a library
routine other than the one the oracle calls, an invariant proved in the paper,
or brute force on tiny inputs.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.linalg
import scipy.special
import torch

from oracle import locks_oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")
D = 128
B = 16


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _rng(seed):
    return np.random.default_rng(seed)


def _pages(rng, n, rank=8, scale=3.0, mean_scale=1.0):
    """Pages with a per-page low-rank structure plus a little noise."""
    out = np.empty((n, B, D))
    for p in range(n):
        U = np.linalg.qr(rng.standard_normal((D, rank)))[0]
        c = rng.standard_normal((B, rank)) * scale * (0.7 ** np.arange(rank))
        out[p] = mean_scale * rng.standard_normal(D) + c @ U.T + 0.05 * rng.standard_normal((B, D))
    return out


# ---------------------------------------------------------------- payload (App. C.1)

def test_payload_bytes_match_paper_table():
    g = _gold("payload_table.json")
    kv = g["geometry"]["kv_bytes_per_page_bf16"]
    assert O.kv_bytes_per_page(2) == kv
    N, b = 1 << 20, 2048
    n_pages, k = N // B, b // B
    for r_s, pay in g["stored_payload_bytes"].items():
        r = int(r_s)
        assert O.payload_bytes(r) == pay
        alpha = pay / kv
        assert round(alpha, 3) == pytest.approx(g["alpha"][r_s])
        # ceiling 1/alpha as the paper rounds it (10x, 17x, 25x)
        assert abs(1 / alpha - g["read_reduction_ceiling"][r_s]) < 0.8
        dense = n_pages * kv
        locks = n_pages * pay + k * kv
        assert round(dense / locks, 1) == pytest.approx(g["reduction_at_1M_b2048"][r_s])
        assert round(100 * n_pages * pay / locks) == g["summary_share_of_read_at_1M_percent"][r_s]
    # logical payload without scales: d*r/2 + B*r + d = 768 B, 9.4 % at r = 8
    logical = D * 8 // 2 + B * 8 + D
    assert logical == g["logical_payload_r8_bytes"]
    assert round(100 * logical / kv, 1) == g["logical_payload_r8_percent"]
    # the abstract's "about 1/10 at r=8 and 1/25 at r=2"
    assert abs(kv / O.payload_bytes(8) - 10) < 0.1 and abs(kv / O.payload_bytes(2) - 25) < 0.2


def test_encoded_record_uses_exactly_the_payload():
    rng = _rng(1)
    for r in (2, 4, 8):
        pk = _pages(rng, 3, rank=8)
        f = O.build_factors(pk, r)
        rec = O.encode(f["mu"], f["V"], f["C"])
        assert rec.shape[1] == O.record_stride(r) and rec.shape[1] % 16 == 0
        assert np.all(rec[:, O.payload_bytes(r):] == 0)   # only padding past the payload


# ---------------------------------------------------------------- exact log-mass

def test_exact_lse_envelope_worked_example():
    """Lemma 'Envelope content-blindness' proof: equal-extreme pages P, P' with
    q = (e1+e2)/sqrt2 have s_P = log B and s_P' = log(B-2 + e^x + e^-x), x = c sqrt2 / sqrt d."""
    for c in (0.5, 3.0, 40.0):
        P = np.zeros((B, D))
        P[0, :2] = (c, -c)
        P[1, :2] = (-c, c)
        Pp = np.zeros((B, D))
        Pp[0, :2] = (c, c)
        Pp[1, :2] = (-c, -c)
        q = np.zeros((1, D))
        q[0, :2] = 1 / math.sqrt(2)
        x = c * math.sqrt(2) / math.sqrt(D)
        sP = O.exact_page_lse(q, P)[0, 0]
        sPp = O.exact_page_lse(q, Pp)[0, 0]
        assert sP == pytest.approx(math.log(B), abs=1e-12)
        assert sPp == pytest.approx(math.log(B - 2 + math.exp(x) + math.exp(-x)), rel=1e-12)
        # both pages have rank-1 deviations, so a rank-1 summary is exact (Prop. score error)
        for page, want in ((P, sP), (Pp, sPp)):
            f = O.build_factors(page[None], 1)
            assert O.score(q, f["mu"], f["V"], f["C"])[0, 0] == pytest.approx(want, abs=1e-12)
        # the envelope score sum_c max(q_c u_c, q_c l_c) is identical for both pages
        env = [np.sum(np.maximum(q[0] * pg.max(0), q[0] * pg.min(0))) for pg in (P, Pp)]
        assert env[0] == pytest.approx(env[1])


def test_exact_lse_partial_page_and_library():
    rng = _rng(2)
    L = 16 * 5 + 7
    keys = rng.standard_normal((L, D)) * 2
    q = rng.standard_normal((3, D))
    s = O.exact_page_lse(q, keys)
    assert s.shape == (3, 6)
    t = torch.from_numpy(q) @ torch.from_numpy(keys).T / math.sqrt(D)
    for j in range(6):
        want = torch.logsumexp(t[:, 16 * j:min(L, 16 * j + 16)], dim=1).numpy()
        np.testing.assert_allclose(s[:, j], want, rtol=0, atol=1e-12)


# ---------------------------------------------------------------- build (Sec. 4 "Build")

def test_build_matches_svd_eckart_young():
    """Cor. 'per-page basis is residual-optimal': captured energy and residual equal the
    truncated SVD of the centred page; V orthonormal; c_i = V^T delta_i."""
    rng = _rng(3)
    pk = _pages(rng, 20, rank=12)
    for r in (1, 2, 4, 8, 15):
        f = O.build_factors(pk, r)
        for p in range(pk.shape[0]):
            Dm = pk[p] - pk[p].mean(0)
            sv = scipy.linalg.svd(Dm, compute_uv=False, lapack_driver="gesvd")
            np.testing.assert_allclose(np.sqrt(f["sigma2"][p, :15]), sv[:15], rtol=1e-9, atol=1e-9)
            V, C = f["V"][p], f["C"][p]
            kept = int(f["kept"][p])
            np.testing.assert_allclose(V[:, :kept].T @ V[:, :kept], np.eye(kept), atol=1e-10)
            np.testing.assert_allclose(C, Dm @ V, atol=1e-9)
            resid = np.sum((Dm - C @ V.T) ** 2)
            assert resid == pytest.approx(np.sum(sv[r:] ** 2), rel=1e-8, abs=1e-9)
            assert np.sum(C ** 2) == pytest.approx(np.sum(sv[:r] ** 2), rel=1e-10)


def test_build_full_rank_reconstructs_keys():
    rng = _rng(4)
    pk = _pages(rng, 6, rank=15)
    f = O.build_factors(pk, 15)
    rec = f["mu"][:, None, :] + np.einsum("pil,pcl->pic", f["C"], f["V"])
    np.testing.assert_allclose(rec, pk, atol=1e-9)


def test_isotropic_null_matches_paper():
    """App. B: rank-8 captured fraction over 20,000 isotropic 16x128 pages."""
    g = _gold("isotropic_null.json")
    rng = _rng(0)
    fr = []
    for chunk in range(g["pages"] // 2000):
        pk = rng.standard_normal((2000, B, D))
        f = O.build_factors(pk, g["rank"])
        fr.append(f["sigma2"][:, :g["rank"]].sum(1) / f["sigma2"].sum(1))
    fr = np.concatenate(fr)
    assert abs(np.median(fr) - g["median"]) <= 2 * g["printed_precision"]["median"]
    assert abs(np.mean(fr) - g["mean"]) <= 2 * g["printed_precision"]["mean"]
    assert abs(np.std(fr) - g["std"]) <= 2 * g["printed_precision"]["std"]


def test_identical_keys_drop_every_mode():
    """Zero modes are dropped (Sec. 4): identical keys give D = 0 and hat s = q^T mu / sqrt d + log B = s."""
    rng = _rng(5)
    k = rng.standard_normal(D) * 3
    page = np.tile(k, (B, 1))
    q = rng.standard_normal((4, D))
    f = O.build_factors(page[None], 8)
    assert f["kept"][0] == 0 and np.all(f["V"] == 0) and np.all(f["C"] == 0)
    want = q @ k / math.sqrt(D) + math.log(B)
    np.testing.assert_allclose(O.score(q, f["mu"], f["V"], f["C"])[:, 0], want, atol=1e-12)
    np.testing.assert_allclose(O.exact_page_lse(q, page)[:, 0], want, atol=1e-12)
    # through the stored record: the centroid is the only nonzero field
    dec = O.decode(O.encode(f["mu"], f["V"], f["C"]), 8)
    want_q = q @ dec["mu"][0] / math.sqrt(D) + math.log(B)
    np.testing.assert_allclose(O.score(q, dec["mu"], dec["V"], dec["C"])[:, 0], want_q, atol=1e-12)


def test_prop_blind_perturbation_is_seen_by_refit():
    """Prop. 'Shared scope is content-blind': +-c u with u orthogonal to a shared W leaves
    every shared sketch unchanged while exact masses separate; a refit per-page basis
    (full rank) tracks the exact mass."""
    rng = _rng(6)
    W = np.linalg.qr(rng.standard_normal((D, 48)))[0]
    u = rng.standard_normal(D)
    u -= W @ (W.T @ u)
    u /= np.linalg.norm(u)
    page = _pages(rng, 1, rank=6)[0]
    q = (0.5 * u + 0.1 * rng.standard_normal(D))[None]
    prev = None
    for c in (0.0, 10.0, 40.0, 160.0):
        P2 = page.copy()
        P2[3] += c * u
        P2[9] -= c * u
        np.testing.assert_allclose(P2 @ W, page @ W, atol=1e-9)            # sketches unchanged
        np.testing.assert_allclose(P2.mean(0), page.mean(0), atol=1e-12)   # centroid unchanged
        s = O.exact_page_lse(q, P2)[0, 0]
        f = O.build_factors(P2[None], 15)
        assert O.score(q, f["mu"], f["V"], f["C"])[0, 0] == pytest.approx(s, abs=1e-9)
        if prev is not None:
            assert s > prev
        prev = s
    assert prev - O.exact_page_lse(q, page)[0, 0] > 4.0


# ---------------------------------------------------------------- score (Eq. 1) and its error bound

def test_full_rank_score_is_exact():
    """Prop. 'Score error characterization': r >= rank(D) gives hat s = s."""
    rng = _rng(7)
    pk = _pages(rng, 12, rank=15, mean_scale=3.0)
    q = rng.standard_normal((5, D)) * 1.5
    f = O.build_factors(pk, 15)
    got = O.score(q, f["mu"], f["V"], f["C"])
    want = O.exact_page_lse(q, pk.reshape(-1, D))
    np.testing.assert_allclose(got, want, atol=1e-10)


def test_score_error_bound_chain():
    """|hat s - s| <= max_i |q_perp^T delta_perp_i| / sqrt d <= |q_perp| sigma_{r+1} / sqrt d
    <= |q_perp| sqrt(tau_r) / sqrt d, for unquantised summaries at any r."""
    rng = _rng(8)
    pk = _pages(rng, 30, rank=12, scale=4.0)
    q = rng.standard_normal((4, D)) * 2
    exact = O.exact_page_lse(q, pk.reshape(-1, D))
    for r in (1, 2, 4, 8):
        f = O.build_factors(pk, r)
        est = O.score(q, f["mu"], f["V"], f["C"])
        for p in range(pk.shape[0]):
            Dm = pk[p] - pk[p].mean(0)
            sv = np.linalg.svd(Dm, compute_uv=False)
            V = f["V"][p]
            resid = Dm - Dm @ V @ V.T
            for g in range(q.shape[0]):
                qp = q[g] - V @ (V.T @ q[g])
                err = abs(est[g, p] - exact[g, p])
                b1 = np.max(np.abs(resid @ qp)) / math.sqrt(D)
                b2 = np.linalg.norm(qp) * sv[r] / math.sqrt(D)
                b3 = np.linalg.norm(qp) * math.sqrt(np.sum(sv[r:] ** 2)) / math.sqrt(D)
                assert err <= b1 + 1e-10
                assert b1 <= b2 + 1e-10
                assert b2 <= b3 + 1e-10
        assert np.max(np.abs(est - exact)) > 1e-6   # the bound is not vacuous here


# ---------------------------------------------------------------- encode / decode

def test_quantize_roundtrip_error_bound():
    rng = _rng(9)
    for r in (2, 4, 8):
        pk = _pages(rng, 40, rank=8, scale=5.0, mean_scale=4.0)
        f = O.build_factors(pk, r)
        dec = O.decode(O.encode(f["mu"], f["V"], f["C"]), r)
        vs, cs, ms = dec["vscale"], dec["cscale"], dec["mscale"]
        # |x - code * s| <= s/2, plus the clamp slack when the f16 scale rounded down
        slack = 1 + 2 * 7 * 2.0 ** -11
        assert np.all(np.abs(dec["V"] - f["V"]) <= vs[:, None, :] / 2 * slack + 1e-12)
        assert np.all(np.abs(dec["C"] - f["C"]) <= cs[:, :, None] / 2 * slack + 1e-12)
        assert np.all(np.abs(dec["mu"] - f["mu"]) <= ms[:, None] / 2 * slack + 1e-12)
        assert dec["vcodes"].min() >= -7 and dec["vcodes"].max() <= 7
        assert np.abs(dec["ccodes"]).max() <= 127 and np.abs(dec["mcodes"]).max() <= 127
        # scales are max|x| / qmax rounded to float16
        np.testing.assert_array_equal(vs, (np.abs(f["V"]).max(1) / 7).astype(np.float16).astype(np.float64))


def test_record_byte_layout_by_hand():
    """A hand-written record: one basis entry, one coefficient, one centroid entry."""
    r = 2
    V = np.zeros((1, D, r))
    C = np.zeros((1, B, r))
    mu = np.zeros((1, D))
    V[0, 5, 1] = 0.5        # column 1, row 5 -> code +7, scale 0.5/7
    V[0, 4, 1] = -0.25      # same byte, low nibble: code rint(-3.5) = -4 (ties to even)
    C[0, 3, 0] = -2.0       # row 3 -> code -127 with scale 2/127
    mu[0, 127] = 1.0        # centroid -> code 127
    rec = O.encode(mu, V, C)[0]
    s_v = np.float16(0.5 / 7)
    assert rec[64 * 1 + 2] == ((-4 + 8) | ((7 + 8) << 4))       # bytes of column 1, rows 4, 5
    assert np.all(rec[0:64] == 8 | (8 << 4))                   # column 0 is all-zero codes
    assert rec[64 * r + 3 * r + 0] == -127 + 128
    assert rec[64 * r + B * r + 127] == 127 + 128
    sc = rec[80 * r + 128:80 * r + 128 + 2 * (r + 17)].view("<f2")
    assert sc[1] == s_v and sc[0] == 0 and sc[r + 3] == np.float16(2.0 / 127)
    assert sc[r + 16] == np.float16(1.0 / 127)


# ---------------------------------------------------------------- combine + select

def _coverage_lib(q, keys, pages, Bp=16):
    """gamma_S(q) from scipy's softmax over every token (pages of Bp tokens)."""
    z = q @ keys.T / math.sqrt(D)
    p = scipy.special.softmax(z, axis=1)
    idx = np.concatenate([np.arange(Bp * j, min(keys.shape[0], Bp * j + Bp)) for j in pages])
    return p[:, idx].sum(1)


@pytest.mark.parametrize("G,Bp", [(1, 16), (2, 16), (4, 16), (2, 32), (4, 64)])
def test_select_matches_brute_force(G, Bp):
    """Cor. 'Group-shared selection': with exact shares, sink + recent + top-(k-2) by mbar
    maximises the group-mean coverage over all k-sets containing sink and recent
    (pages of 16, 32 or 64 tokens)."""
    for seed in range(12):
        rng = _rng(100 + seed)
        n = int(rng.integers(4, 10))
        k = int(rng.integers(2, n))
        keys = rng.standard_normal((Bp * n, D)) * rng.uniform(0.5, 3.0, size=(Bp * n, 1))
        keys[:Bp] *= rng.uniform(0.2, 3.0)      # sink mass varies across heads
        q = rng.standard_normal((G, D)) * rng.uniform(0.5, 2.5, size=(G, 1))
        s = O.exact_page_lse(q, keys, B=Bp)
        sel = O.select_pages(s, n, k)
        best, best_set = -1.0, None
        for rest in itertools.combinations(range(1, n - 1), k - 2):
            S = sorted((0, n - 1) + rest)
            val = _coverage_lib(q, keys, S, Bp).mean()
            if val > best + 1e-12:
                best, best_set = val, S
        assert _coverage_lib(q, keys, sel["ids"], Bp).mean() == pytest.approx(best, abs=1e-12)
        if sel["gap"] > 1e-9:
            assert sel["ids"] == best_set
        # the share-average key of each page is the group-mean coverage of that page
        # alone (scipy softmax over every token), and the ranking gap is the log ratio
        # of the weakest kept candidate to the strongest candidate left out of the
        # brute-force optimum
        share = np.array([_coverage_lib(q, keys, [j], Bp).mean() for j in range(n)])
        np.testing.assert_allclose(sel["log_mbar"], np.log(share), atol=1e-12, rtol=0)
        if k >= 3:
            kept = [j for j in best_set if 0 < j < n - 1]
            left = [j for j in range(1, n - 1) if j not in best_set]
            want_gap = math.log(min(share[kept])) - math.log(max(share[left]))
            assert sel["gap"] == pytest.approx(want_gap, abs=1e-12)
        else:
            assert sel["gap"] == math.inf


def test_select_gap_and_share_keys_by_hand():
    """Values worked out by hand from the share-average combine (Sec. 4 "Score") and
    the gap reading (log mbar of the (k-2)-th minus the (k-1)-th best candidate,
    natural log).  An off-by-one in the cut index, a dropped -log G, a log base
    other than e or a normaliser over the candidates only fails one of these."""
    # G = 1, six complete pages with masses 1, 4, 2, 8, 3, 5 (Z = 23); k = 4 keeps
    # two candidates of pages 1..4: page 3 (8/23) and page 1 (4/23); the next is
    # page 4 (3/23), so the gap is ln(4/3).
    s = np.log(np.array([[1.0, 4.0, 2.0, 8.0, 3.0, 5.0]]))
    sel = O.select_pages(s, 6, 4)
    assert sel["ids"] == [0, 1, 3, 5]
    np.testing.assert_allclose(sel["log_mbar"], np.log(np.array([1, 4, 2, 8, 3, 5]) / 23.0),
                               atol=1e-14, rtol=0)
    assert sel["gap"] == pytest.approx(math.log(4.0 / 3.0), abs=1e-14)
    # k = 5 keeps three (8, 4, 3 of 23); the next candidate holds 2/23: gap ln(3/2)
    sel = O.select_pages(s, 6, 5)
    assert sel["ids"] == [0, 1, 3, 4, 5]
    assert sel["gap"] == pytest.approx(math.log(1.5), abs=1e-14)
    # G = 2 with unequal normalisers.  Head 0 masses 1, 1, 1, 1, 1, 1 (Z = 6), head 1
    # masses 1, 1/6, 1/3, 1/2, 2, 1/12 (Z = 49/12).
    # Shares: head 0 all 1/6; head 1 (12/49)(1, 1/6, 1/3, 1/2, 2, 1/12)
    #       = 12/49, 2/49, 4/49, 6/49, 24/49, 1/49.
    # mbar = (1/2)(1/6 + head-1 share):
    #   page 0: (49 + 72) / 588 = 121/588      page 1: (49 + 12) / 588 = 61/588
    #   page 2: (49 + 24) / 588 = 73/588       page 3: (49 + 36) / 588 = 85/588
    #   page 4: (49 + 144) / 588 = 193/588     page 5: (49 + 6) / 588 = 55/588
    # (they sum to 1).  Candidates 1..4 ranked: 4, 3, 2, 1.  k = 4 keeps pages 4
    # and 3; gap = ln(85/73).
    h1 = np.array([1.0, 1 / 6, 1 / 3, 1 / 2, 2.0, 1 / 12])
    s2 = np.log(np.stack([np.ones(6), h1]))
    want = np.log(np.array([121, 61, 73, 85, 193, 55]) / 588.0)
    sel = O.select_pages(s2, 6, 4)
    np.testing.assert_allclose(sel["log_mbar"], want, atol=1e-14, rtol=0)
    assert sel["ids"] == [0, 3, 4, 5]
    assert sel["gap"] == pytest.approx(math.log(85 / 73), abs=1e-14)
    # adding a constant to one head's scores changes neither shares nor table
    sel_shift = O.select_pages(s2 + np.array([[3.0], [-7.0]]), 6, 4)
    np.testing.assert_allclose(sel_shift["log_mbar"], want, atol=1e-13, rtol=0)
    # G = 4, seven pages with a partial recent page (n = 7, six summarised): heads
    # 0..3 are heads 0 and 1 above, twice, with page 6 carrying no score, so
    # mbar of the summarised pages is as above and the candidates are pages 1..5;
    # k = 3 keeps page 4 (193/588) against page 3 (85/588): gap ln(193/85).
    s4 = np.concatenate([s2, s2])
    sel = O.select_pages(s4, 7, 3)
    np.testing.assert_allclose(sel["log_mbar"], want, atol=1e-14, rtol=0)
    assert sel["ids"] == [0, 4, 6]
    assert sel["gap"] == pytest.approx(math.log(193 / 85), abs=1e-14)
    # an exact tie at the cut: pages 1 and 2 share one key; k = 3 keeps page 1
    # (lower index) and the gap is 0
    st = np.log(np.array([[5.0, 2.0, 2.0, 1.0]]))
    sel = O.select_pages(st, 4, 3)
    assert sel["ids"] == [0, 1, 3] and sel["gap"] == 0.0
    # no cut: k = 2 keeps sink and recent only; n <= k keeps everything
    assert O.select_pages(s, 6, 2)["gap"] == math.inf
    assert O.select_pages(s, 6, 2)["ids"] == [0, 5]
    assert O.select_pages(s, 6, 6)["gap"] == math.inf


def test_select_g1_is_plain_ranking_and_small_n():
    rng = _rng(11)
    s = rng.standard_normal((1, 50))
    sel = O.select_pages(s, 50, 10)
    order = [j for j in np.argsort(-s[0], kind="stable") if j not in (0, 49)][:8]
    assert sel["ids"] == sorted([0, 49] + order)
    assert O.select_pages(s[:, :7], 8, 10)["ids"] == list(range(8))     # n <= k: everything
    assert O.select_pages(np.zeros((1, 0)), 1, 2)["ids"] == [0]          # one partial page
    assert O.select_pages(np.zeros((1, 0)), 0, 2)["ids"] == []          # empty sequence
    # ties go to the lower page index
    flat = np.zeros((1, 20))
    assert O.select_pages(flat, 20, 5)["ids"] == [0, 1, 2, 3, 19]


def test_retention_bound_theorem():
    """Thm. 'Retention of the group-shared selection' (ii): the table chosen from
    unquantised estimates keeps >= e^{-4 eta} of the exact-share table's group coverage."""
    for seed in range(6):
        rng = _rng(200 + seed)
        n, G, k = 40, 4, 8
        pk = _pages(rng, n, rank=12, scale=4.0)
        keys = pk.reshape(-1, D)
        q = rng.standard_normal((G, D)) * 2
        exact = O.exact_page_lse(q, keys)
        f = O.build_factors(pk, 2)
        est = O.score(q, f["mu"], f["V"], f["C"])
        eta = np.max(np.abs(est - exact))
        S_est = O.select_pages(est, n, k)["ids"]
        S_ex = O.select_pages(exact, n, k)["ids"]
        cov_est = _coverage_lib(q, keys, S_est).mean()
        cov_ex = _coverage_lib(q, keys, S_ex).mean()
        assert cov_est >= math.exp(-4 * eta) * cov_ex - 1e-12
        # robustness corollary on a single query, Delta = eta, always-kept pages included
        g0 = O.select_pages(est[:1], n, k)["ids"]
        e0 = O.select_pages(exact[:1], n, k)["ids"]
        assert _coverage_lib(q[:1], keys, g0)[0] >= math.exp(-2 * eta) * _coverage_lib(q[:1], keys, e0)[0] - 1e-12


# ---------------------------------------------------------------- attention

def test_dense_matches_torch_sdpa():
    rng = _rng(12)
    for L in (1, 15, 16, 100, 1000):
        keys = rng.standard_normal((L, D)) * 2
        vals = rng.standard_normal((L, D))
        q = rng.standard_normal((4, D))
        o, lse = O.dense_step(q, keys, vals)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q)[None, :, None, :], torch.from_numpy(keys)[None, None].expand(1, 4, L, D),
            torch.from_numpy(vals)[None, None].expand(1, 4, L, D))[0, :, 0]
        np.testing.assert_allclose(o, ref.numpy(), atol=1e-12)
        z = torch.from_numpy(q) @ torch.from_numpy(keys).T / math.sqrt(D)
        np.testing.assert_allclose(lse, torch.logsumexp(z, 1).numpy(), atol=1e-12)


def test_budget_covering_everything_is_dense():
    rng = _rng(13)
    L = 16 * 9 + 5
    keys = rng.standard_normal((L, D)) * 2
    vals = rng.standard_normal((L, D))
    q = rng.standard_normal((2, D))
    rec = O.unit_summaries(keys, 4)
    res = O.decode_step(q, keys, vals, rec, 4, budget_tokens=L + 16)
    o, lse = O.dense_step(q, keys, vals)
    assert res["ids"] == list(range(10))
    np.testing.assert_allclose(res["out"], o, atol=1e-12)
    np.testing.assert_allclose(res["lse"], lse, atol=1e-12)
    assert np.isnan(res["sel_lse"][:, 9]).all()          # the partial page has no summary


def test_truncation_identity_and_bound():
    """Lemma 'Coverage, the exact deficit': o - o_S = eps (vbar_{S^c} - vbar_S) exactly and
    |o - o_S| <= 2 R (1 - gamma_S)."""
    rng = _rng(14)
    n = 12
    keys = rng.standard_normal((16 * n, D)) * 2
    vals = rng.standard_normal((16 * n, D))
    q = rng.standard_normal((3, D))
    R = np.max(np.linalg.norm(vals, axis=1))
    for S in ([0, 11], [0, 3, 5, 11], list(range(n))):
        o, _ = O.dense_step(q, keys, vals)
        oS, _ = O.attend(q, keys, vals, S)
        p = scipy.special.softmax(q @ keys.T / math.sqrt(D), axis=1)
        mask = np.zeros(16 * n, bool)
        for j in S:
            mask[16 * j:16 * j + 16] = True
        gam = p[:, mask].sum(1)
        eps = 1 - gam
        vS = (p[:, mask] @ vals[mask]) / gam[:, None]
        if (~mask).any():
            vC = (p[:, ~mask] @ vals[~mask]) / eps[:, None]
            np.testing.assert_allclose(o - oS, eps[:, None] * (vC - vS), atol=1e-12)
        else:
            np.testing.assert_allclose(o, oS, atol=1e-12)
        assert np.all(np.linalg.norm(o - oS, axis=1) <= 2 * R * (1 - gam) + 1e-12)
        np.testing.assert_allclose(O.coverage(q, keys, S), gam, atol=1e-12)


def test_empty_and_partial_sequences():
    rng = _rng(15)
    q = rng.standard_normal((2, D))
    empty = np.zeros((0, D))
    res = O.decode_step(q, empty, empty, np.zeros((0, O.record_stride(8)), np.uint8), 8, 64)
    assert res["ids"] == [] and np.all(res["out"] == 0) and np.all(res["lse"] == -np.inf)
    for L in (1, 7, 16, 17, 33):
        keys = rng.standard_normal((L, D))
        vals = rng.standard_normal((L, D))
        rec = O.unit_summaries(keys, 8)
        assert rec.shape[0] == L // 16
        res = O.decode_step(q, keys, vals, rec, 8, 48)
        o, lse = O.dense_step(q, keys, vals)        # n <= k = 3 always here
        np.testing.assert_allclose(res["out"], o, atol=1e-12)


# ---------------------------------------------------------------- basis precision variants
# (Sec. 5 "Ablations": int8 and bf16 bases; the r8fp control of the retention remark)

def test_bf16_rounding_matches_torch():
    """The oracle's round-to-nearest-even bfloat16 against torch's conversion."""
    rng = _rng(40)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 4, 20000),
                        [0.0, -0.0, 1.0, -1.0, 1.00390625, 1.01171875, 3.0e38]])
    want = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy()
    np.testing.assert_array_equal(O.bf16_round(x).astype(np.int16), want)
    np.testing.assert_array_equal(O.bf16_value(O.bf16_round(x)),
                                  torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16)
                                  .to(torch.float64).numpy())


@pytest.mark.parametrize("basis", ["int8", "bf16"])
def test_variant_record_roundtrip(basis):
    """Every field decodes to its value within its rounding error (int8: s/2 of the
    column scale; bf16: the unit roundoff 2^-8); coefficients and centroid are the same
    int8 codes as in the int4 record, and the record holds exactly its payload."""
    rng = _rng(41)
    pk = _pages(rng, 12)
    f = O.build_factors(pk, 8)
    rec = O.encode(f["mu"], f["V"], f["C"], basis)
    dec = O.decode(rec, 8, basis)
    if basis == "int8":
        s = dec["vscale"][:, None, :]
        assert np.all(np.abs(dec["V"] - f["V"]) <= s / 2 + 1e-12)
        assert np.all(np.abs(dec["vcodes"]) <= 127)
        amax = np.max(np.abs(f["V"]), axis=1)
        assert np.allclose(dec["vscale"], (amax / 127).astype(np.float16).astype(np.float64))
    else:
        # unit roundoff of bfloat16 (8 significant bits): |x - bf16(x)| <= 2^-8 |x|
        assert np.all(np.abs(dec["V"] - f["V"]) <= np.abs(f["V"]) * 2.0 ** -8 * 1.0001 + 1e-30)
        assert np.all(dec["vscale"] == 1.0)
    ref = O.decode(O.encode(f["mu"], f["V"], f["C"]), 8)
    np.testing.assert_array_equal(dec["ccodes"], ref["ccodes"])
    np.testing.assert_array_equal(dec["mcodes"], ref["mcodes"])
    used = O.payload_bytes(8, basis=basis)
    assert np.all(rec[:, used:] == 0) and rec.shape[1] == O.record_stride(8, basis)
    # the basis occupies d * r elements of 1 (int8) or 2 (bf16) bytes
    assert used - O.payload_bytes(8) == D * 8 * (O.BASIS_BYTES[basis] - 0.5)


def test_basis_precision_orders_score_error():
    """The finer the basis, the closer the stored score is to the unquantised one (the
    ablation's ordering): int4 > int8 > bf16 in mean |error|, and a bf16 basis with
    an exact (unquantised) C and mu is within bf16 rounding of the fp64 score."""
    rng = _rng(42)
    pk = _pages(rng, 200, scale=4.0)
    f = O.build_factors(pk, 8)
    q = rng.standard_normal((4, D))
    exact = O.score(q, f["mu"], f["V"], f["C"])
    err = {}
    for basis in ("int4", "int8", "bf16"):
        dec = O.decode(O.encode(f["mu"], f["V"], f["C"], basis), 8, basis)
        err[basis] = np.mean(np.abs(O.score(q, dec["mu"], dec["V"], dec["C"]) - exact))
    assert err["int4"] > 2 * err["int8"] and err["int8"] > err["bf16"], err
    Vb = O.bf16_value(O.bf16_round(f["V"]))
    zb = O.score(q, f["mu"], Vb, f["C"])
    # |dz| <= sum_l |c_l| |q . dv_l| / sqrt d <= r |C|max |q| 2^-8 / sqrt d (|dv_l| <= 2^-8 |v_l| = 2^-8)
    bound = np.max(np.linalg.norm(q, axis=1)) * np.max(np.abs(f["C"])) * 8 * 2.0 ** -8 / math.sqrt(D)
    assert np.max(np.abs(zb - exact)) <= bound


# --------------------------------------------------------------------------
# KIVI fake quantisation at page finalize (Sec. 5 "KV-cache quantization under
# extreme sparsity"; App. C full-grid protocol)
# --------------------------------------------------------------------------

def test_kivi_worked_examples_by_hand():
    """Asymmetric 2-bit min/max on hand-computed slices: min 0, max 15 gives scale
    5 and reconstruction 5 * rint(x / 5) (ties to even at 2.5 and 7.5); an offset
    slice keeps its zero point; a negative slice works from its minimum."""
    x = np.array([0, 1, 2, 2.5, 3, 7, 7.5, 8, 12, 13, 15], dtype=np.float32)
    want = np.array([0, 0, 0, 0, 5, 5, 10, 10, 10, 15, 15], dtype=np.float32)
    np.testing.assert_array_equal(O.kivi_fake_quant(x, 2, axis=0), want)
    np.testing.assert_array_equal(O.kivi_fake_quant(x + 100, 2, axis=0), want + 100)
    # from the minimum -15: (x + 15) / 5 = 3, 2.8, 2.6, 2.5, 2.4, 1.6, 1.5, 1.4, 0.6,
    # 0.4, 0 rounds to 3, 3, 3, 2, 2, 2, 2, 1, 1, 0, 0 (2.5 and 1.5 to even)
    np.testing.assert_array_equal(O.kivi_fake_quant(-x, 2, axis=0), np.array(
        [0, 0, 0, -5, -5, -5, -5, -10, -10, -15, -15], dtype=np.float32))
    # 4 bits on 0..15: every integer is a level, nothing moves
    t = np.arange(16, dtype=np.float32)
    np.testing.assert_array_equal(O.kivi_fake_quant(t, 4, axis=0), t)
    # 2^b - 1 levels above the minimum, not 2^b: 3 bits on 0..14 step 2 is exact
    np.testing.assert_array_equal(O.kivi_fake_quant(2 * t[:8], 3, axis=0), 2 * t[:8])


def test_kivi_page_axes_keys_per_channel_values_per_token_group():
    """Keys that are constant along tokens (different per channel) and values that
    are constant inside each 32-channel group of a token pass unchanged; the
    transposed arrangement does not."""
    rng = np.random.default_rng(5)
    chan = O.bf16_value(O.bf16_round(rng.normal(size=128) * 3))
    keys = np.tile(chan, (16, 1))
    tok = O.bf16_value(O.bf16_round(rng.normal(size=(16, 4)) * 3))
    vals = np.repeat(tok, 32, axis=1)
    kq, vq = O.kivi_page(keys, vals, 2, 32)
    np.testing.assert_array_equal(kq, keys)
    np.testing.assert_array_equal(vq, vals)
    kq2, vq2 = O.kivi_page(vals[:, :128], keys, 2, 32)
    assert np.any(kq2 != vals) and np.any(vq2 != keys)


@pytest.mark.parametrize("bits", [2, 4, 8])
@pytest.mark.parametrize("g", [16, 32, 128])
def test_kivi_levels_extremes_and_error_bound(bits, g):
    """Per slice: at most 2^b distinct values, minimum and maximum reproduced
    exactly (bf16 inputs), and every value within half a step plus half a bf16
    unit of the result."""
    rng = np.random.default_rng(bits * 1000 + g)
    keys = O.bf16_value(O.bf16_round(rng.normal(size=(16, 128)) * 2 + rng.normal(size=128)))
    vals = O.bf16_value(O.bf16_round(rng.normal(size=(16, 128))))
    kq, vq = O.kivi_page(keys, vals, bits, g)
    for orig, out in ((keys.T, kq.T), (vals.reshape(-1, g), vq.reshape(-1, g))):
        for a, b in zip(orig, out):
            assert len(np.unique(b)) <= 2 ** bits
            assert b.min() == a.min() and b.max() == a.max()
            step = (a.max() - a.min()) / (2 ** bits - 1)
            tol = step / 2 * (1 + 1e-5) + np.abs(b) * 2.0 ** -8
            assert np.all(np.abs(b - a) <= tol)


# ---------------------------------------------------------------- page size (App. D.3)

def test_page_size_payload_fractions_match_paper():
    """App. D.3: at r = 8 the logical summary falls from 9.4% of the page's KV bytes at
    B = 16 to 5.5% and 3.5% at B = 32 and 64; the budget buys k = ceil(b / B) pages,
    two of them free at b = 256, B = 64."""
    g = _gold("page_size.json")
    r = g["rank"]
    for B_s, pct in g["logical_payload_percent"].items():
        Bp = int(B_s)
        logical = O.logical_payload_bytes(r, B=Bp)
        assert logical == D * r // 2 + Bp * r + D
        assert round(100 * logical / O.kv_bytes_per_page(2, B=Bp), 1) == pct
        # the stored record adds r + B + 1 float16 scales
        assert O.payload_bytes(r, B=Bp) == logical + 2 * (r + Bp + 1)
        assert O.record_stride(r, B=Bp) % 16 == 0
    # b = 256 at B = 64: k = 4 pages, sink and recent take two, two are chosen
    rng = _rng(61)
    keys = rng.standard_normal((64 * 20 + 5, D))
    vals = rng.standard_normal((64 * 20 + 5, D))
    q = rng.standard_normal((2, D))
    rec = O.unit_summaries(keys, 8, B=64)
    st = O.decode_step(q, keys, vals, rec, 8, 256, B=64)
    assert len(st["ids"]) == 4 and st["ids"][0] == 0 and st["ids"][-1] == 20
    assert len(st["ids"]) - 2 == g["free_pages_at_b256_B64"]


def _pages_B(rng, n, Bp, rank=8, scale=3.0):
    out = np.empty((n, Bp, D))
    for p in range(n):
        U = np.linalg.qr(rng.standard_normal((D, rank)))[0]
        c = rng.standard_normal((Bp, rank)) * scale * (0.7 ** np.arange(rank))
        out[p] = rng.standard_normal(D) + c @ U.T + 0.05 * rng.standard_normal((Bp, D))
    return out


@pytest.mark.parametrize("Bp", [32, 64])
def test_page_size_build_matches_svd(Bp):
    """Cor. 'per-page basis is residual-optimal' on B x B Grams: energies and residuals
    equal the truncated SVD of the centred page; exact reconstruction at full rank."""
    rng = _rng(62 + Bp)
    pk = _pages_B(rng, 6, Bp, rank=12)
    for r in (2, 8, 15):
        f = O.build_factors(pk, r)
        for p in range(pk.shape[0]):
            Dm = pk[p] - pk[p].mean(0)
            sv = scipy.linalg.svd(Dm, compute_uv=False, lapack_driver="gesvd")
            np.testing.assert_allclose(np.sqrt(f["sigma2"][p, :Bp - 1]), sv[:Bp - 1], rtol=1e-8,
                                       atol=1e-8)
            V, C = f["V"][p], f["C"][p]
            np.testing.assert_allclose(V.T @ V, np.eye(r), atol=1e-10)
            np.testing.assert_allclose(C, Dm @ V, atol=1e-9)
            resid = np.sum((Dm - C @ V.T) ** 2)
            assert resid == pytest.approx(np.sum(sv[r:] ** 2), rel=1e-8, abs=1e-9)
    full = O.build_factors(pk, Bp - 1)
    rec = full["mu"][:, None, :] + np.einsum("pil,pcl->pic", full["C"], full["V"])
    np.testing.assert_allclose(rec, pk, atol=1e-9)
    # full rank: the reconstructed page score is the exact page log-mass of B tokens,
    # itself the log-sum-exp of its 16-token halves (scipy)
    q = rng.standard_normal((3, D)) * 1.5
    got = O.score(q, full["mu"], full["V"], full["C"])
    want = O.exact_page_lse(q, pk.reshape(-1, D), B=Bp)
    np.testing.assert_allclose(got, want, atol=1e-10)
    halves = O.exact_page_lse(q, pk.reshape(-1, D), B=16).reshape(3, -1, Bp // 16)
    np.testing.assert_allclose(want, scipy.special.logsumexp(halves, axis=2), atol=1e-12)


@pytest.mark.parametrize("Bp", [32, 64])
def test_page_size_record_layout_and_roundtrip(Bp):
    """The record of a B-token page: [basis r x 64 B][coefficients B x r][centroid
    128][float16 scales: r basis, B coefficient rows, 1 centroid][padding];
    decoding restores every entry within half a quantisation step."""
    rng = _rng(70 + Bp)
    r = 4
    pk = _pages_B(rng, 5, Bp)
    f = O.build_factors(pk, r)
    rec = O.encode(f["mu"], f["V"], f["C"])
    assert rec.shape[1] == O.record_stride(r, B=Bp)
    dec = O.decode(rec, r, B=Bp)
    assert np.all(np.abs(dec["V"] - f["V"]) <= dec["vscale"][:, None, :] / 2 + 1e-12)
    assert np.all(np.abs(dec["C"] - f["C"]) <= dec["cscale"][:, :, None] / 2 + 1e-12)
    assert np.all(np.abs(dec["mu"] - f["mu"]) <= dec["mscale"][:, None] / 2 + 1e-12)
    # the same bytes read by hand
    p = 2
    coef = rec[p, 64 * r:64 * r + Bp * r].astype(np.int64) - 128
    np.testing.assert_array_equal(coef.reshape(Bp, r), dec["ccodes"][p])
    mu = rec[p, 64 * r + Bp * r:64 * r + Bp * r + 128].astype(np.int64) - 128
    np.testing.assert_array_equal(mu, dec["mcodes"][p])
    sc = rec[p, 64 * r + Bp * r + 128:64 * r + Bp * r + 128 + 2 * (r + Bp + 1)].view("<f2")
    np.testing.assert_array_equal(sc[r:r + Bp].astype(np.float64), dec["cscale"][p])
    assert np.all(rec[:, O.payload_bytes(r, B=Bp):] == 0)


@pytest.mark.parametrize("Bp", [32, 64])
def test_page_size_attention_and_dense(Bp):
    """A B-token page is B consecutive tokens: attention over page j at page size B
    equals attention over its 16-token pages; a budget covering every page is dense
    attention."""
    rng = _rng(80 + Bp)
    L = Bp * 9 + 7
    keys = rng.standard_normal((L, D))
    vals = rng.standard_normal((L, D))
    q = rng.standard_normal((4, D))
    sub = Bp // 16
    for pages in ([0], [3, 9], [1, 2, 5, 9]):
        o1, l1 = O.attend(q, keys, vals, pages, B=Bp)
        small = [sub * j + i for j in pages for i in range(sub) if 16 * (sub * j + i) < L]
        o2, l2 = O.attend(q, keys, vals, small, B=16)
        np.testing.assert_allclose(o1, o2, atol=1e-12)
        np.testing.assert_allclose(l1, l2, atol=1e-12)
    rec = O.unit_summaries(keys, 8, B=Bp)
    st = O.decode_step(q, keys, vals, rec, 8, Bp * 10, B=Bp)
    o_d, l_d = O.dense_step(q, keys, vals)
    assert st["ids"] == list(range(10))
    np.testing.assert_allclose(st["out"], o_d, atol=1e-12)
    np.testing.assert_allclose(st["lse"], l_d, atol=1e-12)
