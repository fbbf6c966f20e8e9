"""CPU fp64 oracle of the Locks per-step sparse decode attention.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path (the HIP
library and its binding) never calls it and shares no code with it.

Everything is plain NumPy in float64, one definition per function, in the order
the paper states it:

* decode attention, page-level coverage and the exact page log-mass
  (Sec. 2 "Decode-time attention"; Lemma 1 in the coverage appendix);
* the per-page build -- centre, B x B Gram eigendecomposition, rank-r truncation,
  zero modes dropped (Sec. 4 "Build");
* the stored summary: int4 basis, int8 coefficients and centroid, per-column /
  per-row scales, stored payload 818 / 490 / 326 bytes (Sec. 4 "Build";
  App. C.1 budget-accounting table);
* the reconstructed page score of Eq. (1) (Sec. 4 "Score");
* the share-average GQA combine and the shared top-k table with the sink and most
  recent page always kept (Sec. 4 "Score"; Cor. "Group-shared selection");
* exact attention restricted to the selected pages (Sec. 2; App. E).

Readings of points the paper leaves open:

* scale 1/sqrt(d) in both the score and attention;
* a mode is dropped when sigma^2 <= max(ZERO_MODE_REL * sigma_1^2,
  ZERO_MODE_ABS * mean_i |k_i|^2): relative to the leading mode, and absolutely
  against the page's mean squared key norm so that rounding residue of an
  all-equal page never counts as a mode;
* quantisation is symmetric with float16 scales: basis columns |code| <= 7,
  coefficient rows and the centroid |code| <= 127; scale = f16(max|x| / qmax)
  (clamped to the largest finite float16), code = clamp(rint(x / scale)) with
  ties to even, scale 0 => codes 0;
* pages hold B = 16 tokens unless stated; B = 32 and 64 are the page sizes of
  App. D.3 "Page size", where the budget buys k = ceil(b / B) pages;
* byte layout (one record per (physical block, KV head)):
  [basis: r columns x 64 bytes, column l holds d=128 excess-8 nibbles, element c
  in byte c//2, low nibble for even c][coefficients: B x r excess-128 bytes,
  row-major][centroid: 128 excess-128 bytes][float16 scales: r basis-column,
  B coefficient-row, 1 centroid][zero padding to a multiple of 16 bytes];
* basis precision variants (the ablation of Sec. 5 "Ablations" and the r8fp
  control of the retention remark): an int8 basis stores each column as 128
  excess-128 bytes with one float16 scale f16(max|v| / 127); a bf16 basis stores
  each column as 128 little-endian bfloat16 values (round to nearest even) and
  its column-scale slots hold 1.0.  Coefficients and centroid stay int8 and the
  field order is unchanged;
* KV quantisation at page finalize (Sec. 5 "KV-cache quantization under extreme
  sparsity", the KIVI composition, and the protocol of its full grid in App. C):
  fake quantisation, i.e. quantise then dequantise back to bfloat16 in place,
  asymmetric min/max with 2^b levels: keys per channel over the page's 16 tokens,
  values per token over groups of g consecutive channels (g = 32 unless stated).
  scale s = (max - min) / (2^b - 1), code = min(rint((x - min) / s), 2^b - 1),
  x' = bf16(code * s + min); every operation is one float32 rounding (the
  kernel's precision, which decides the codes), the result rounded to bfloat16
  to nearest even; a group with s = 0 is left as it is.  POST builds a page's
  summary from the keys as written and then quantises the page; PRE quantises
  first and builds from the quantised keys;
* sign convention: each basis column's largest-magnitude entry (first on ties)
  is made positive, the matching coefficient column flipped with it;
* the normaliser Z_g of the share sums every page that has a summary (complete
  pages, sink and recent included); candidates exclude the sink (page 0) and the
  most recent page (the one holding the last token); ties go to the lower page
  index; if the sequence has at most k pages every page is selected;
* an empty sequence attends nothing: output 0, log-sum-exp -inf.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Tuple

import numpy as np

PAGE = 16          # B, tokens per page
HEAD_DIM = 128     # d
ZERO_MODE_REL = 1e-6
ZERO_MODE_ABS = 1e-10
F16_MAX = 65504.0
INT4_MAX = 7
INT8_MAX = 127


# --------------------------------------------------------------------------
# Summary payload accounting (Sec. 4 "Build"; App. C.1 table)
# --------------------------------------------------------------------------

BASIS_BYTES = {"int4": 0.5, "int8": 1, "bf16": 2}   # bytes per basis element


def payload_bytes(r: int, d: int = HEAD_DIM, B: int = PAGE, basis: str = "int4") -> int:
    """Stored bytes per page: the d*r basis (int4 by default) + B*r int8 + d int8
    + 2-byte scales for r basis columns, B coefficient rows and the centroid."""
    return logical_payload_bytes(r, d, B, basis) + 2 * (r + B + 1)


def logical_payload_bytes(r: int, d: int = HEAD_DIM, B: int = PAGE, basis: str = "int4") -> int:
    """The summary's entries without their scales: d*r basis entries (int4 by
    default) plus B*r + d int8 bytes (Sec. 4 "Build"; App. D.3 "Page size")."""
    return int(d * r * BASIS_BYTES[basis]) + B * r + d


def record_stride(r: int, basis: str = "int4", B: int = PAGE) -> int:
    p = payload_bytes(r, B=B, basis=basis)
    return (p + 15) // 16 * 16


def kv_bytes_per_page(elem_bytes: int = 2, d: int = HEAD_DIM, B: int = PAGE) -> int:
    return 2 * B * d * elem_bytes


# --------------------------------------------------------------------------
# Exact quantities (Sec. 2; coverage appendix, Lemma 1)
# --------------------------------------------------------------------------

def _lse(x: np.ndarray, axis: int = -1) -> np.ndarray:
    """log(sum(exp(x))) along an axis, max-shifted; -inf when everything is -inf."""
    m = np.max(x, axis=axis, keepdims=True)
    m_safe = np.where(np.isfinite(m), m, 0.0)
    s = np.sum(np.exp(x - m_safe), axis=axis, keepdims=True)
    with np.errstate(divide="ignore"):
        out = np.log(s) + m_safe
    return np.squeeze(out, axis=axis)


def logits(q: np.ndarray, keys: np.ndarray) -> np.ndarray:
    """q [G][d], keys [T][d] -> q^T k / sqrt(d), shape [G][T]."""
    return (q @ keys.T) / math.sqrt(keys.shape[1])


def exact_page_lse(q: np.ndarray, keys: np.ndarray, n_pages: Optional[int] = None,
                   B: int = PAGE) -> np.ndarray:
    """s_j(q) = log sum_{i in P_j} exp(q^T k_i / sqrt d) for pages of B tokens.

    q [G][d], keys [L][d]; returns [G][n] over the pages that hold tokens
    (a partial last page uses its valid tokens only)."""
    L = keys.shape[0]
    n = (L + B - 1) // B if n_pages is None else n_pages
    z = logits(q, keys)
    out = np.empty((q.shape[0], n))
    for j in range(n):
        out[:, j] = _lse(z[:, j * B:min(L, (j + 1) * B)], axis=1)
    return out


def attend(q: np.ndarray, keys: np.ndarray, vals: np.ndarray,
           pages: Optional[List[int]] = None, B: int = PAGE) -> Tuple[np.ndarray, np.ndarray]:
    """Softmax attention of each query over the tokens of the given pages of B
    tokens (all tokens when pages is None), renormalised over that set.

    Returns (o [G][d], lse [G]) with lse the log of the softmax denominator."""
    L = keys.shape[0]
    G = q.shape[0]
    if pages is None:
        idx = np.arange(L)
    else:
        idx = np.concatenate([np.arange(j * B, min(L, (j + 1) * B)) for j in pages]
                             ) if len(pages) else np.zeros(0, dtype=np.int64)
    if idx.size == 0:
        return np.zeros((G, vals.shape[1] if vals.ndim == 2 else HEAD_DIM)), np.full(G, -np.inf)
    z = logits(q, keys[idx])
    lse = _lse(z, axis=1)
    p = np.exp(z - lse[:, None])
    return p @ vals[idx], lse


def coverage(q: np.ndarray, keys: np.ndarray, pages: List[int], B: int = PAGE) -> np.ndarray:
    """gamma_S(q): share of the full softmax mass that falls in pages S, per query."""
    s = exact_page_lse(q, keys, B=B)
    tot = _lse(s, axis=1)
    sel = _lse(s[:, pages], axis=1) if len(pages) else np.full(q.shape[0], -np.inf)
    return np.exp(sel - tot)


# --------------------------------------------------------------------------
# Build (Sec. 4 "Build")
# --------------------------------------------------------------------------

def build_factors(page_keys: np.ndarray, r: int) -> Dict[str, np.ndarray]:
    """Per-page rank-r factors for a stack of pages.

    page_keys [P][B][d].  For each page: mu = mean of its keys, D = K - 1 mu^T,
    eigendecompose the B x B Gram D D^T = U S^2 U^T with eigenvalues descending,
    keep the r leading modes, drop zero modes (coefficients and basis column 0),
    V = D^T U_r S_r^{-1} (orthonormal columns) and C = U_r S_r (c_i = V^T delta_i).

    Returns mu [P][d], V [P][d][r], C [P][B][r], sigma2 [P][B] (all eigenvalues,
    descending, clipped at 0) and kept [P] (number of nonzero kept modes)."""
    K = np.asarray(page_keys, dtype=np.float64)
    P, Bt, d = K.shape
    mu = K.mean(axis=1)
    D = K - mu[:, None, :]
    gram = D @ np.transpose(D, (0, 2, 1))
    w, U = np.linalg.eigh(gram)                  # ascending
    w = w[:, ::-1]
    U = U[:, :, ::-1]
    w = np.maximum(w, 0.0)
    rr = min(r, Bt)
    lam = w[:, :rr]
    top = w[:, :1]
    energy = np.mean(np.sum(K * K, axis=2), axis=1)[:, None]
    floor = np.maximum(ZERO_MODE_REL * top, ZERO_MODE_ABS * energy)
    keep = (lam > floor) & (lam > 0.0)                  # descending => a prefix
    sig = np.sqrt(np.where(keep, lam, 1.0))
    Ur = U[:, :, :rr]
    V = np.zeros((P, d, r))
    C = np.zeros((P, Bt, r))
    V[:, :, :rr] = np.where(keep[:, None, :], np.einsum("pic,pil->pcl", D, Ur) / sig[:, None, :], 0.0)
    C[:, :, :rr] = np.where(keep[:, None, :], Ur * sig[:, None, :], 0.0)
    # sign convention: the largest-magnitude entry of each basis column is positive
    j = np.argmax(np.abs(V), axis=1)                           # [P][r], first on ties
    lead = np.take_along_axis(V, j[:, None, :], axis=1)[:, 0, :]
    flip = np.where(lead < 0, -1.0, 1.0)
    V = V * flip[:, None, :]
    C = C * flip[:, None, :]
    kept = keep.sum(axis=1)
    return {"mu": mu, "V": V, "C": C, "sigma2": w, "kept": kept}


# --------------------------------------------------------------------------
# Summary encoding (Sec. 4 "Build": int4 basis, int8 coefficients and centroid,
# per-column and per-row scales; stored payload from App. C.1)
# --------------------------------------------------------------------------

def _f16(x: np.ndarray) -> np.ndarray:
    return np.minimum(np.asarray(x, dtype=np.float64), F16_MAX).astype(np.float16)


def quantize(x: np.ndarray, qmax: int, axis) -> Tuple[np.ndarray, np.ndarray]:
    """Symmetric quantisation with one float16 scale per slice along `axis`.

    Returns integer codes in [-qmax, qmax] and the float16 scales."""
    amax = np.max(np.abs(x), axis=axis, keepdims=True)
    s16 = _f16(amax / qmax)
    s = s16.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        codes = np.where(s > 0, np.clip(np.rint(x / np.where(s > 0, s, 1.0)), -qmax, qmax), 0.0)
    return codes.astype(np.int64), np.squeeze(s16, axis=axis)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 (ties to even) of float32(x), as uint16 bit patterns."""
    u = np.asarray(x, dtype=np.float64).astype(np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_value(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)


def encode(mu: np.ndarray, V: np.ndarray, C: np.ndarray, basis: str = "int4") -> np.ndarray:
    """Quantise and pack one summary per page: mu [P][d], V [P][d][r], C [P][B][r]
    -> uint8 records [P][record_stride(r, basis)]."""
    P, d, r = V.shape
    B = C.shape[1]                                    # tokens per page
    assert d == HEAD_DIM
    cq, cs = quantize(C, INT8_MAX, axis=2)            # per coefficient row (token)
    mq, ms = quantize(mu, INT8_MAX, axis=1)           # one centroid scale
    out = np.zeros((P, record_stride(r, basis, B)), dtype=np.uint8)
    cb = int(d * BASIS_BYTES[basis])                  # bytes per basis column
    if basis == "int4":
        vq, vs = quantize(V, INT4_MAX, axis=1)        # per basis column
        nib = (vq + 8).astype(np.uint8)               # excess-8, [P][d][r]
        for l in range(r):
            col = nib[:, :, l]
            out[:, cb * l:cb * l + cb] = col[:, 0::2] | (col[:, 1::2] << 4)
    elif basis == "int8":
        vq, vs = quantize(V, INT8_MAX, axis=1)
        for l in range(r):
            out[:, cb * l:cb * l + cb] = (vq[:, :, l] + 128).astype(np.uint8)
    elif basis == "bf16":
        bits = bf16_round(V)                          # [P][d][r]
        for l in range(r):
            out[:, cb * l:cb * l + cb] = bits[:, :, l].astype("<u2").view(np.uint8).reshape(P, cb)
        vs = np.ones((P, r), dtype=np.float16)
    else:
        raise ValueError(basis)
    off = cb * r
    out[:, off:off + B * r] = (cq + 128).astype(np.uint8).reshape(P, B * r)
    off += B * r
    out[:, off:off + d] = (mq + 128).astype(np.uint8)
    off += d
    scales = np.concatenate([vs.reshape(P, r), cs.reshape(P, B), ms.reshape(P, 1)], axis=1)
    out[:, off:off + 2 * (r + B + 1)] = scales.astype("<f2").view(np.uint8).reshape(P, -1)
    return out


def decode(records: np.ndarray, r: int, basis: str = "int4", B: int = PAGE) -> Dict[str, np.ndarray]:
    """Inverse of `encode` for pages of B tokens: uint8 [P][stride] -> fp64 mu [P][d],
    V [P][d][r], C [P][B][r]
    (code times float16 scale; bf16 basis values as stored), plus the raw codes."""
    rec = np.asarray(records, dtype=np.uint8)
    P = rec.shape[0]
    d = HEAD_DIM
    cb = int(d * BASIS_BYTES[basis])
    vcodes = np.zeros((P, d, r), dtype=np.int64)
    vvals = None
    for l in range(r):
        b = rec[:, cb * l:cb * l + cb]
        if basis == "int4":
            b = b.astype(np.int64)
            vcodes[:, 0::2, l] = (b & 15) - 8
            vcodes[:, 1::2, l] = (b >> 4) - 8
        elif basis == "int8":
            vcodes[:, :, l] = b.astype(np.int64) - 128
        else:
            if vvals is None:
                vvals = np.zeros((P, d, r))
            vvals[:, :, l] = bf16_value(b.copy().view("<u2"))
    off = cb * r
    ccodes = rec[:, off:off + B * r].astype(np.int64).reshape(P, B, r) - 128
    off += B * r
    mcodes = rec[:, off:off + d].astype(np.int64) - 128
    off += d
    sc = rec[:, off:off + 2 * (r + B + 1)].copy().view("<f2").astype(np.float64)
    vs, cs, ms = sc[:, :r], sc[:, r:r + B], sc[:, r + B]
    V = vvals * vs[:, None, :] if basis == "bf16" else vcodes * vs[:, None, :]
    return {"mu": mcodes * ms[:, None], "V": V, "C": ccodes * cs[:, :, None],
            "vcodes": vcodes, "ccodes": ccodes, "mcodes": mcodes,
            "vscale": vs, "cscale": cs, "mscale": ms}


# --------------------------------------------------------------------------
# Score, Eq. (1) (Sec. 4 "Score")
# --------------------------------------------------------------------------

def score(q: np.ndarray, mu: np.ndarray, V: np.ndarray, C: np.ndarray) -> np.ndarray:
    """hat s_j(q) = log sum_i exp[(q^T mu_j + (V_j^T q)^T c_i) / sqrt d].

    q [G][d]; mu [P][d], V [P][d][r], C [P][B][r] -> [G][P]."""
    d = q.shape[1]
    a = q @ mu.T                                      # [G][P]
    p = np.einsum("gc,pcl->gpl", q, V)               # [G][P][r] = V_j^T q
    z = (a[:, :, None] + np.einsum("gpl,pil->gpi", p, C)) / math.sqrt(d)
    return _lse(z, axis=2)


# --------------------------------------------------------------------------
# Share-average combine and shared top-k table (Sec. 4 "Score";
# Cor. "Group-shared selection"; App. E union table)
# --------------------------------------------------------------------------

def select_pages(s_hat: np.ndarray, n_pages: int, k: int) -> Dict[str, object]:
    """Shared page table for one (sequence, KV head).

    s_hat [G][n_c]: page scores of the n_c complete (summarised) pages.
    Every page holding a token is one of n_pages; the sink is page 0 and the
    most recent page is n_pages - 1.  With m_g(j) = e^{s_gj} / sum_j' e^{s_gj'}
    and mbar_j = mean_g m_g(j), the table holds the sink, the most recent page and
    the k-2 other pages of largest mbar (lower index first on ties), ascending.

    Returns ids (list, ascending), log_mbar [n_c] and the ranking gap
    log mbar_(k-2) - log mbar_(k-1) among the candidates (inf if no cut)."""
    G, n_c = s_hat.shape
    if n_pages <= 0:
        return {"ids": [], "log_mbar": np.zeros(0), "gap": math.inf}
    if n_c > 0:
        lz = _lse(s_hat, axis=1)                      # log Z_g over summarised pages
        log_mbar = _lse(s_hat - lz[:, None], axis=0) - math.log(G)
    else:
        log_mbar = np.zeros(0)
    if n_pages <= k:
        return {"ids": list(range(n_pages)), "log_mbar": log_mbar, "gap": math.inf}
    cand = list(range(1, n_pages - 1))
    order = sorted(cand, key=lambda j: (-log_mbar[j], j))
    top = order[:k - 2]
    gap = float(log_mbar[order[k - 3]] - log_mbar[order[k - 2]]) if k >= 3 else math.inf
    ids = sorted(set([0, n_pages - 1] + top))
    return {"ids": ids, "log_mbar": log_mbar, "gap": gap}


# --------------------------------------------------------------------------
# KIVI fake quantisation of a finalised page (Sec. 5 "KV-cache quantization
# under extreme sparsity"; App. C full-grid protocol)
# --------------------------------------------------------------------------

def kivi_fake_quant(x: np.ndarray, bits: int, axis) -> np.ndarray:
    """Asymmetric b-bit min/max quantise-dequantise of every slice of the float32
    array x along `axis` (one scale and zero point per slice), float32 throughout;
    returns the float32 values before the final bfloat16 rounding."""
    x = np.asarray(x, dtype=np.float32)
    levels = np.float32(2 ** bits - 1)
    mn = np.min(x, axis=axis, keepdims=True)
    mx = np.max(x, axis=axis, keepdims=True)
    s = (mx - mn) / levels                                  # float32 / float32
    live = s > 0
    safe = np.where(live, s, np.float32(1.0))
    code = np.minimum(np.rint((x - mn) / safe), levels)     # ties to even
    y = code * safe + mn                                    # two float32 roundings
    return np.where(live, y, x).astype(np.float32)


def kivi_page(keys: np.ndarray, vals: np.ndarray, bits: int, v_group: int = 32):
    """One finalised page [B][d] of keys and of values, bfloat16 in and out (as
    float64 arrays of bfloat16 values): keys per channel over the page's tokens,
    values per token over groups of v_group channels."""
    kq = kivi_fake_quant(keys, bits, axis=0)
    B, d = vals.shape
    vq = kivi_fake_quant(np.asarray(vals).reshape(B, d // v_group, v_group), bits,
                         axis=2).reshape(B, d)
    return bf16_value(bf16_round(kq)), bf16_value(bf16_round(vq))


# --------------------------------------------------------------------------
# One decode step for one (sequence, KV head)
# --------------------------------------------------------------------------

def pages_of(keys: np.ndarray, B: int = PAGE) -> Tuple[np.ndarray, int, int]:
    """Split [L][d] keys into complete pages [n_c][B][d]; returns (pages, n_c, n)."""
    L = keys.shape[0]
    n_c = L // B
    n = (L + B - 1) // B
    return keys[:n_c * B].reshape(n_c, B, keys.shape[1]), n_c, n


def unit_summaries(keys: np.ndarray, r: int, basis: str = "int4", B: int = PAGE) -> np.ndarray:
    """Encoded summaries [n_c][stride] of the complete B-token pages of one
    (sequence, KV head)."""
    pk, n_c, _ = pages_of(keys, B)
    if n_c == 0:
        return np.zeros((0, record_stride(r, basis, B)), dtype=np.uint8)
    f = build_factors(pk, r)
    return encode(f["mu"], f["V"], f["C"], basis)


def decode_step(q: np.ndarray, keys: np.ndarray, vals: np.ndarray, records: np.ndarray,
                r: int, budget_tokens: int, basis: str = "int4", B: int = PAGE) -> Dict[str, object]:
    """Score every summarised page from its decoded record, select the shared table,
    attend over it.  records [n_c][stride] are the complete pages' summaries; pages
    hold B tokens and the page budget is k = ceil(b / B) (App. D.3 "Page size")."""
    L = keys.shape[0]
    n_c, n = L // B, (L + B - 1) // B
    k = (budget_tokens + B - 1) // B
    dec = decode(records[:n_c], r, basis, B) if n_c else None
    s_hat = score(q, dec["mu"], dec["V"], dec["C"]) if n_c else np.zeros((q.shape[0], 0))
    sel = select_pages(s_hat, n, k)
    o, lse = attend(q, keys, vals, sel["ids"], B)
    sel_lse = np.full((q.shape[0], k), np.nan)
    for t, j in enumerate(sel["ids"]):
        if j < n_c:
            sel_lse[:, t] = s_hat[:, j]
    return {"s_hat": s_hat, "ids": sel["ids"], "gap": sel["gap"], "log_mbar": sel["log_mbar"],
            "out": o, "lse": lse, "sel_lse": sel_lse}


def dense_step(q: np.ndarray, keys: np.ndarray, vals: np.ndarray):
    """Dense decode attention over every token (the same-GPU baseline's definition)."""
    return attend(q, keys, vals, None)
