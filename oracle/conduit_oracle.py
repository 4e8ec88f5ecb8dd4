"""Conduit refresh step: plain float64 CPU oracle.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The HIP product path
never calls, links or imports it, and this module imports nothing from the
product package.

It computes, slowly and in float64, what the paper defines for one refresh
step over reused visual KV caches:

  * Eq. 1-2 (Sec. 3.1)      visual-token sets, image map pi(t), budget k;
  * Eq. 6  (Sec. 3.3)       query- and head-mean cached-key attention a_t;
  * Eq. 7  (Sec. 3.3)       value-norm proxy ||V_t|| and multi-layer score s_t;
  * Eq. 8-9 (Sec. 3.4)      image means g_j, cross-image mean, coefficients c_j;
  * Eq. 10-11 (Sec. 3.5)    composite score s_hat and one global top-k;
  * Algorithm 1 (App. A.1)  the order of these steps and the k = 0 exit;
  * Eq. 3 and App. D.1/D.3 the residual value-write error left by a refresh set:
    isotropic Monte Carlo displacements and the projected error;
  * selective recompute (Sec. 3, Sec. 4.1 cache-reuse protocol): the selected
    visual rows get their fresh K/V written into the cache, unselected rows are
    reused stale, and each selected row attends causally over that merged
    prefix.

Readings of points the paper leaves open (labels used below):
  R1  the scoring softmax normalises over the span token's full causal row
      (NORM_CAUSAL_ROW); NORM_VISUAL_ONLY renormalises over visual keys only;
  R2  logit scale is passed in (1/sqrt(d) in every workload);
  R3  H in Eq. 6 is the number of query heads; query head h reads KV head
      h // (H_q / H_kv) (grouped-query attention);
  R4  ||V_t|| is taken over the H_kv cached heads concatenated;
  R5  k = floor(r * N_vis) in exact integer arithmetic;
  R6  top-k ties go to the lower visual index;
  R8  if the cross-image mean is 0 every c_j is 1;
  R11 refresh attention of a selected row at position p covers keys 0..p of
      the merged cache, itself included;
  R25 the RMS aggregation (Eq. 4's bar-alpha, the squared-error surrogate)
      runs over the same (span token, query head) set as Eq. 6's mean;
  R26 explicit quotas k_j proportional to c_j n_j (App. D cross-image
      diagnostic): largest-remainder apportionment of k, capped at n_j with
      the surplus re-apportioned, ties to the lower image index; if the
      remaining weights are all zero they fall back to n_j; the arithmetic is
      float32 in image order (floating point decides integers there, so the
      decision is taken in the kernel's precision).  Within an image the k_j
      largest s_t are kept (R6 ties).
  R27 the request's text (every position outside the images: changed prefix,
      separators, span) is processed normally (Sec. 3.1): its rows get fresh
      K/V and attend like the selected visual rows, outside the budget; a
      step's recompute rows are the selected visual positions followed by the
      text positions;
  R29 the isotropic displacement of App. D.1 spans the concatenated cached
      value (R4), so its dimensionality is H_kv * d: xi_t = kappa ||V_t||
      z_t / sqrt(H_kv d) with z_t ~ N(0, I) given as input, hence
      E ||xi_t||^2 = kappa^2 ||V_t||^2;
  R30 the residual of Eq. 3 is evaluated for every span row and query head
      (query head h reads the KV-head-h/G slice of xi) with the cached-key
      attention of R1, the output map taken as the identity (no weights);
      the estimate is the mean over samples, rows and heads.  The projected
      error (App. D.3: stale values set to zero) is the same residual with
      xi_t = V_t;
  R28 a paged cache keeps token t in row t mod P of page table[t div P]
      (block-table KV storage of a serving engine, Sec. 4.3); it holds the same
      logical cache as the contiguous layout, so every result is the same.

Inputs are numpy arrays; bf16 data arrives as raw uint16 bit patterns and is
decoded here (the oracle never sees a value the GPU path produced).
"""
from __future__ import annotations

import numpy as np

NORM_CAUSAL_ROW = 0
NORM_VISUAL_ONLY = 1

# Aggregation of the cached-key attention over span tokens and heads.
AGG_MEAN = 0   # Eq. 6: mean
AGG_RMS = 1    # Eq. 4: root-mean-square (R25)

# Selection rules.
RANK_COMPOSITE = 0   # Eq. 10-11: global top-k of s_t * c_pi(t)
RANK_ATTENTION = 1   # value norm dropped: global top-k of (A_t / |L|) * c_pi(t)
RANK_EXPLICIT = 2    # quotas k_j ~ c_j n_j, then top-k_j of s_t inside image j (R26)


# --------------------------------------------------------------------------
# Inputs
# --------------------------------------------------------------------------

def to_f64(x: np.ndarray) -> np.ndarray:
    """Decode a cache/query array to float64.

    float32/float64 arrays are upcast exactly.  uint16 arrays are bf16 bit
    patterns: the 16 bits are the top half of an IEEE binary32 value.
    """
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def visual_layout(img_pos, img_off):
    """Eq. 1: the visual-token sets V_j and the image map pi(t).

    Image j occupies the contiguous sequence positions
    img_pos[j] .. img_pos[j] + n_j - 1, with n_j = img_off[j+1] - img_off[j];
    visual token t (0 <= t < N_vis) is numbered image by image in sequence
    order.  Returns (P_vis, pi): P_vis[t] is the sequence position of visual
    token t and pi[t] its image index.
    """
    positions, owner = [], []
    for j in range(len(img_pos)):
        n_j = int(img_off[j + 1]) - int(img_off[j])
        for u in range(n_j):
            positions.append(int(img_pos[j]) + u)
            owner.append(j)
    return np.array(positions, dtype=np.int64), np.array(owner, dtype=np.int64)


def budget(n_vis: int, r_num: int, r_den: int) -> int:
    """Eq. 2: k = floor(r * N_vis) with r = r_num / r_den, in integers."""
    return (int(r_num) * int(n_vis)) // int(r_den)


# --------------------------------------------------------------------------
# Scoring pass (Eq. 6, Eq. 7 value norm; Algorithm 1 scoring loop)
# --------------------------------------------------------------------------

def attention_row(q_vec, keys, scale):
    """Softmax attention of one query vector over a set of key rows.

    Returns (alpha, lse): alpha over the given keys, lse = log sum exp of the
    scaled logits (natural log).
    """
    z = scale * (keys @ q_vec)
    m = np.max(z)
    e = np.exp(z - m)
    total = np.sum(e)
    return e / total, m + np.log(total)


def value_norms(v_cache, img_pos, img_off):
    """Eq. 7's value-norm proxy ||V_t|| over the concatenated cached heads
    (R4), for every visual token.  It depends on the cache only, so it can be
    tabulated once when the cache is built (Sec. 4.3) and is exactly the
    norm the scoring pass would read."""
    v_cache = to_f64(v_cache)
    P_vis, _ = visual_layout(img_pos, img_off)
    v_rows = v_cache[P_vis].reshape(len(P_vis), -1)
    return np.sqrt(np.sum(v_rows * v_rows, axis=1))


def score_layer(q, k_cache, v_cache, q_pos0, img_pos, img_off, norm=NORM_CAUSAL_ROW,
                scale=None, agg=AGG_MEAN):
    """One scored layer of the query-conditioned scoring pass.

    q        [n_q, H_q, d]     span queries; span token i sits at q_pos0 + i
    k_cache  [N_ctx, H_kv, d]  the layer's cached keys (stale visual rows)
    v_cache  [N_ctx, H_kv, d]  the layer's cached values
    Returns a [N_vis] (Eq. 6 mean, or Eq. 4's root-mean-square with
    agg=AGG_RMS), v [N_vis] (value-norm proxy of Eq. 7) and the row
    log-sum-exp lse [n_q, H_q] of each softmax (natural log).
    """
    q = to_f64(q)
    k_cache = to_f64(k_cache)
    n_q, n_q_heads, d = q.shape
    n_kv_heads = k_cache.shape[1]
    group = n_q_heads // n_kv_heads
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    P_vis, _ = visual_layout(img_pos, img_off)
    n_vis = len(P_vis)

    col_sum = np.zeros(n_vis)
    lse = np.zeros((n_q, n_q_heads))
    for i in range(n_q):
        p = q_pos0 + i
        for h in range(n_q_heads):
            kv = h // group
            if norm == NORM_CAUSAL_ROW:
                # keys 0..p; visual positions all lie before the span
                alpha, lse[i, h] = attention_row(q[i, h], k_cache[: p + 1, kv, :], scale)
                alpha = alpha[P_vis]
            else:
                alpha, lse[i, h] = attention_row(q[i, h], k_cache[P_vis, kv, :], scale)
            col_sum += alpha if agg == AGG_MEAN else alpha * alpha
    a = col_sum / (n_q * n_q_heads)
    if agg == AGG_RMS:
        a = np.sqrt(a)
    return a, value_norms(v_cache, img_pos, img_off), lse


# --------------------------------------------------------------------------
# Layer aggregation, image reweighting, composite score, top-k
# --------------------------------------------------------------------------

def aggregate_layers(a_layers, v_layers):
    """Eq. 7 and Algorithm 1 score loop.

    Returns (s, A): s_t = (1/|L|) sum_l a_t^(l) v_t^(l), and A_t = sum_l a_t^(l)
    (the per-token attention total that Eq. 8 averages per image).
    """
    n_layers = len(a_layers)
    s = np.zeros_like(np.asarray(a_layers[0], dtype=np.float64))
    A = np.zeros_like(s)
    for a_l, v_l in zip(a_layers, v_layers):
        s += np.asarray(a_l, np.float64) * np.asarray(v_l, np.float64)
        A += np.asarray(a_l, np.float64)
    return s / n_layers, A


def image_coefficients(A, n_layers, img_off, lam):
    """Eq. 8 (g_j and its cross-image mean) and Eq. 9 (c_j).

    A is the per-token attention summed over the scored layers.
    Returns (g, g_bar, c).  If the cross-image mean is zero, c_j = 1 (R8).
    """
    n_images = len(img_off) - 1
    g = np.zeros(n_images)
    for j in range(n_images):
        lo, hi = int(img_off[j]), int(img_off[j + 1])
        g[j] = np.sum(A[lo:hi]) / (n_layers * (hi - lo))
    g_bar = np.sum(g) / n_images
    if g_bar == 0.0:
        return g, g_bar, np.ones(n_images)
    c = (1.0 - lam) + lam * g / g_bar
    return g, g_bar, c


def composite_score(s, c, pi):
    """Eq. 10: s_hat_t = s_t * c_pi(t)."""
    return s * c[pi]


def topk_select(s_hat, k):
    """Eq. 11: the k visual tokens with the largest composite score.

    Ties go to the lower visual index (R6).  Returns the selected visual
    indices in ascending order.
    """
    s_hat = np.asarray(s_hat, dtype=np.float64)
    t = np.arange(len(s_hat))
    order = np.lexsort((t, -s_hat))  # primary key -s_hat, then t
    return np.sort(order[:k])


def refresh_mask(s_hat, k, img_pos, img_off):
    """Algorithm 1 tail: TopK then the binary mask over visual positions.

    Returns (idx, pos, mask): ascending visual indices, their sequence
    positions and the uint8 mask M over visual tokens.
    """
    P_vis, _ = visual_layout(img_pos, img_off)
    mask = np.zeros(len(P_vis), dtype=np.uint8)
    if k == 0:
        return np.zeros(0, np.int64), np.zeros(0, np.int64), mask
    idx = topk_select(s_hat, k)
    mask[idx] = 1
    return idx, P_vis[idx], mask


# --------------------------------------------------------------------------
# Selective recompute: cache merge and refresh attention
# --------------------------------------------------------------------------

def merge_cache(cache, pos, new_rows):
    """Selected rows take their recomputed values; every other row is reused.

    cache [N_ctx, H_kv, d]; pos [k] sequence positions; new_rows [k, H_kv, d].
    Returns (merged, stale_rows): a new array, and the rows it replaced.
    """
    merged = np.array(cache, copy=True)
    stale = np.array(cache[pos], copy=True)
    merged[pos] = new_rows
    return merged, stale


def refresh_attention(q_sel, k_merged, v_merged, pos, scale=None, rows=None):
    """Causal attention of the selected rows over the merged cache (R11).

    q_sel [k, H_q, d]: fresh queries of the selected rows, row i at pos[i].
    Returns (O [k, H_q, d], lse [k, H_q]) in float64; with `rows` given only
    those rows are computed (the others stay zero).
    """
    q_sel = to_f64(q_sel)
    k_merged = to_f64(k_merged)
    v_merged = to_f64(v_merged)
    n_rows, n_q_heads, d = q_sel.shape
    n_kv_heads = k_merged.shape[1]
    group = n_q_heads // n_kv_heads
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((n_rows, n_q_heads, d))
    lse = np.zeros((n_rows, n_q_heads))
    for i in (range(n_rows) if rows is None else rows):
        p = int(pos[i])
        for h in range(n_q_heads):
            kv = h // group
            alpha, lse[i, h] = attention_row(q_sel[i, h], k_merged[: p + 1, kv, :], scale)
            out[i, h] = alpha @ v_merged[: p + 1, kv, :]
    return out, lse


# --------------------------------------------------------------------------
# Algorithm 1 end to end, then the per-layer refresh
# --------------------------------------------------------------------------

def explicit_quotas(c, n, k):
    """R26: quotas k_j proportional to c_j n_j that sum to k, each <= n_j.

    Largest remainder with caps: images whose proportional share reaches n_j
    take n_j and leave the apportionment; the rest share what remains.  All
    arithmetic is float32 in image order.  Returns an int64 array.
    """
    c = np.asarray(c, dtype=np.float32)
    n = np.asarray(n, dtype=np.int64)
    K = len(n)
    quota = np.zeros(K, dtype=np.int64)
    live = np.ones(K, dtype=bool)
    left = int(k)
    while True:
        w = np.array([np.float32(c[j]) * np.float32(n[j]) for j in range(K)], dtype=np.float32)
        total = np.float32(0.0)
        for j in range(K):
            if live[j]:
                total = np.float32(total + w[j])
        if total == np.float32(0.0):  # no weight left: share by size
            w = n.astype(np.float32)
            total = np.float32(0.0)
            for j in range(K):
                if live[j]:
                    total = np.float32(total + w[j])
        share = np.zeros(K, dtype=np.float32)
        for j in range(K):
            if live[j]:
                share[j] = np.float32(np.float32(left) * w[j]) / total
        capped = [j for j in range(K) if live[j] and share[j] >= np.float32(n[j])]
        if not capped:
            break
        for j in capped:
            quota[j] = n[j]
            live[j] = False
            left -= int(n[j])
    base = np.zeros(K, dtype=np.int64)
    frac = np.full(K, -1.0, dtype=np.float32)
    for j in range(K):
        if live[j]:
            base[j] = min(int(np.floor(share[j])), int(n[j]))
            frac[j] = np.float32(share[j] - np.float32(base[j]))
    quota[live] = base[live]
    rest = left - int(base[live].sum())
    # remaining seats to the largest fractional parts, ties to the lower image
    order = sorted((j for j in range(K) if live[j] and quota[j] < n[j]), key=lambda j: (-frac[j], j))
    for j in order[:rest]:
        quota[j] += 1
    return quota


def select_explicit(s, c, img_off, k):
    """R26: quotas from explicit_quotas, then the k_j largest s_t of each
    image (R6 ties).  Returns (quota, ascending visual indices)."""
    n = np.diff(np.asarray(img_off, dtype=np.int64))
    quota = explicit_quotas(c, n, k)
    chosen = []
    for j in range(len(n)):
        lo = int(img_off[j])
        chosen.extend((lo + topk_select(s[lo:lo + int(n[j])], int(quota[j]))).tolist())
    return quota, np.sort(np.asarray(chosen, dtype=np.int64))


def select(layers, q_pos0, img_pos, img_off, k, lam=1.0, norm=NORM_CAUSAL_ROW, scale=None,
           agg=AGG_MEAN, rule=RANK_COMPOSITE, v_tables=None):
    """Algorithm 1: scoring over every scored layer, reweighting, top-k.

    layers: sequence of dicts with 'q', 'k', 'v' (one per scored layer); any
    subset of a model's layers may be passed (|L| = len(layers)).
    v_tables: optional per-layer value-norm tables used instead of the norms
    of the cached V (they are equal by construction, Sec. 4.3).
    Returns a dict with per-layer a, v, lse and the shared s, A, g, c, s_hat,
    idx, pos, mask (and quota for RANK_EXPLICIT).  With k == 0 nothing is
    scored (Algorithm 1 early exit).
    """
    P_vis, pi = visual_layout(img_pos, img_off)
    if k == 0:
        idx, pos, mask = refresh_mask(np.zeros(len(P_vis)), 0, img_pos, img_off)
        return {"idx": idx, "pos": pos, "mask": mask}
    a_l, v_l, lse_l = [], [], []
    for li, layer in enumerate(layers):
        a, v, lse = score_layer(layer["q"], layer["k"], layer["v"], q_pos0, img_pos, img_off,
                                norm=norm, scale=scale, agg=agg)
        if v_tables is not None:
            v = np.asarray(v_tables[li], dtype=np.float64)
        a_l.append(a)
        v_l.append(v)
        lse_l.append(lse)
    s, A = aggregate_layers(a_l, v_l)
    g, g_bar, c = image_coefficients(A, len(layers), img_off, lam)
    out = {"a": a_l, "v": v_l, "lse": lse_l, "s": s, "A": A, "g": g, "g_bar": g_bar, "c": c}
    if rule == RANK_EXPLICIT:
        quota, idx = select_explicit(s, c, img_off, k)
        mask = np.zeros(len(P_vis), dtype=np.uint8)
        mask[idx] = 1
        out.update({"s_hat": composite_score(s, c, pi), "quota": quota, "idx": idx,
                    "pos": P_vis[idx], "mask": mask})
        return out
    base = s if rule == RANK_COMPOSITE else A / len(layers)
    s_hat = composite_score(base, c, pi)
    idx, pos, mask = refresh_mask(s_hat, k, img_pos, img_off)
    out.update({"s_hat": s_hat, "idx": idx, "pos": pos, "mask": mask})
    return out


# --------------------------------------------------------------------------
# Residual value-write error of a refresh set (Eq. 3, App. D.1, App. D.3)
# --------------------------------------------------------------------------

def iso_displacements(v_cache, img_pos, img_off, z, kappa):
    """App. D.1 isotropic staleness samples (R29).

    z [M, N_vis, H_kv, d]: standard normal draws.  Returns
    xi [M, N_vis, H_kv, d] with xi_t = kappa ||V_t|| / sqrt(H_kv d) * z_t.
    """
    z = to_f64(z)
    dim = z.shape[2] * z.shape[3]
    sigma = kappa * value_norms(v_cache, img_pos, img_off) / np.sqrt(dim)
    return sigma[None, :, None, None] * z


def projected_displacements(v_cache, img_pos, img_off):
    """App. D.3: with every stale visual value set to zero, the displacement
    of a non-refreshed token is its value; returns [1, N_vis, H_kv, d]."""
    P_vis, _ = visual_layout(img_pos, img_off)
    return to_f64(v_cache)[P_vis][None]


def residual_error(q, k_cache, q_pos0, img_pos, img_off, refreshed, xi, norm=NORM_CAUSAL_ROW,
                   scale=None):
    """Squared norm of Eq. 3's residual, sum over non-refreshed visual t of
    alpha^c_{q,t} xi_t, for each displacement sample, span row and query head
    (R30).

    refreshed [N_vis]: nonzero for tokens in the refresh set T.
    xi [M, N_vis, H_kv, d].  Returns err [M, n_q, H_q].
    """
    q = to_f64(q)
    k_cache = to_f64(k_cache)
    xi = np.asarray(xi, dtype=np.float64)
    n_q, n_q_heads, d = q.shape
    group = n_q_heads // k_cache.shape[1]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    P_vis, _ = visual_layout(img_pos, img_off)
    keep = np.asarray(refreshed) == 0
    err = np.zeros((xi.shape[0], n_q, n_q_heads))
    for i in range(n_q):
        p = q_pos0 + i
        for h in range(n_q_heads):
            kv = h // group
            if norm == NORM_CAUSAL_ROW:
                alpha, _ = attention_row(q[i, h], k_cache[: p + 1, kv, :], scale)
                alpha = alpha[P_vis]
            else:
                alpha, _ = attention_row(q[i, h], k_cache[P_vis, kv, :], scale)
            alpha = np.where(keep, alpha, 0.0)
            for m in range(xi.shape[0]):
                y = alpha @ xi[m, :, kv, :]
                err[m, i, h] = y @ y
    return err


def iso_estimate(err):
    """App. D.1's estimate: the mean of the sampled squared residuals (over
    samples, span rows and query heads, R30)."""
    return float(np.mean(err))


# --------------------------------------------------------------------------
# Text rows and paged caches
# --------------------------------------------------------------------------

def text_positions(n_ctx, img_pos, img_off):
    """Positions 0..n_ctx-1 that hold no visual token: the request's text,
    processed normally (Sec. 3.1, R27)."""
    P_vis, _ = visual_layout(img_pos, img_off)
    is_visual = np.zeros(int(n_ctx), dtype=bool)
    is_visual[P_vis] = True
    return np.flatnonzero(~is_visual).astype(np.int64)


def recompute_rows(sel_pos, text_pos):
    """The rows one layer recomputes: selected visual rows, then text rows
    (R27)."""
    return np.concatenate([np.asarray(sel_pos, np.int64), np.asarray(text_pos, np.int64)])


def paged_to_contiguous(pages, block_table, n_ctx):
    """The logical cache a page pool holds (R28).

    pages [n_pages, P, H_kv, d]; block_table[i] is the page of tokens
    i*P .. i*P + P - 1.  Returns [n_ctx, H_kv, d].
    """
    pages = np.asarray(pages)
    P = pages.shape[1]
    out = np.empty((int(n_ctx),) + pages.shape[2:], dtype=pages.dtype)
    for t in range(int(n_ctx)):
        out[t] = pages[int(block_table[t // P]), t % P]
    return out


def refresh_layer(k_cache, v_cache, pos, k_new, v_new, q_sel, scale=None, rows=None):
    """Selective recompute of one layer: merge, then refresh attention.

    Returns (k_merged, v_merged, O, lse).  With no selected rows the cache is
    returned unchanged and O is empty (the cache-reuse anchor).
    """
    k_cache = to_f64(k_cache)
    v_cache = to_f64(v_cache)
    if len(pos) == 0:
        d = k_cache.shape[2]
        return k_cache, v_cache, np.zeros((0, 0, d)), np.zeros((0, 0))
    k_m, _ = merge_cache(k_cache, pos, to_f64(k_new))
    v_m, _ = merge_cache(v_cache, pos, to_f64(v_new))
    out, lse = refresh_attention(q_sel, k_m, v_m, pos, scale=scale, rows=rows)
    return k_m, v_m, out, lse
