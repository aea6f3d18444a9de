"""CPU oracle of Fusion's staged adaptive ViT inference (merge -> exit -> prune).

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it; the GPU library and its
Python binding never do.  It shares no code with the HIP path.

Plain, slow and per sample: every sample runs Algorithm 1 (Sec. III-B) on its
own token list, so ragged lengths are natural and no compaction exists here.
float32 NumPy throughout (BLAS sgemm for the matrix products), integer counts
in IEEE double with the expressions written below.

Precision modes
  ``fp32``    no rounding at all.
  ``bf16emu`` still float32 arithmetic, but values are rounded to bfloat16
              (round to nearest even) exactly where the bf16 GPU path stores
              them: every matrix-product weight, every matrix-product left
              operand (patches, LN outputs, attention output, GELU output),
              q/k/v, and the un-normalised attention probabilities before
              they multiply V.  Everything else (accumulation, bias, residual
              stream, LN statistics, softmax sums, router, similarities,
              merge arithmetic, token sizes, CLS scores) stays float32.

Readings of the paper where it is silent (each also listed in the design doc):
  token order: CLS first, patches in raster order, patch vectors in
      (channel, ky, kx) order; learned position embedding added (Eq. 1).
  block: pre-norm, LN eps 1e-6, qkv bias, scale dh^-1/2, exact-erf GELU
      (Eq. 2).
  proportional attention: scores += ln(size of key token), the companion of
      size-weighted merging (Sec. III-C builds on ToMe's matching).
  merge: cosine similarity of the float32 hidden states after the block;
      only patch tokens take part; A = even, B = odd current patch slots;
      argmax ties -> lowest B slot; top-r by best similarity, ties -> lowest
      A slot; dst <- (s_dst x_dst + sum_asc s_a x_a) / (s_dst + sum_asc s_a);
      sizes and CLS scores add; survivors keep their order (Sec. III-C).
  merge count, rule "budget": r = clamp(floor(2 rho m r_b + 1/2), 0,
      floor(N/2)) with m = sigmoid(w . z_cls + beta) (Eq. 4); rho is the
      profile ratio of Eq. 5 and 2 r_b replaces the candidate count N_b/2,
      so that a neutral router (m = 1/2) merges exactly rho * r_b pairs.
  merge count, rule "fraction" (Sec. III-C as written): m~ = rho m (Eq. 5),
      r = min(floor(m~ N / 2), floor(N/2)), the doubles formed in the order
      ((rho m) N) / 2.
  exit heads (kind per exit block): "linear" = LN + linear on the CLS
      token; "cls_mlp" = LN, linear to the hidden width, exact GELU, linear
      to C, on the CLS token; "pool_mlp" = the same MLP on the size-weighted
      mean of the patch tokens sum_t s_t z_t / sum_t s_t (CLS excluded; a
      sample without patch tokens pools to the zero vector), taken after the
      block's merge (Sec. IV-I, Parameter and Memory Overhead).
  exit: head_b as above, c = max softmax
      = 1 / sum_k exp(l_k - l_max); exit iff delta < 1 and c >= delta
      (Eq. 6-7).  Exited samples return head_b's logits.
  prune: score, rule "cls_attn" = head-mean CLS attention probability of
      block b (added up through block b's merge); rule "learned" = the
      linear scorer s_i = w . z_i + beta on the hidden states after the
      merge (Eq. 8); keep CLS + top floor(tau' N) patch tokens,
      tau' = min(1, max(0, 1 - rho (1 - tau_b))), ties -> lower position,
      order kept; only samples that did not exit (Eq. 8, Sec. III-B).

Decision margins (in O(1) units) are logged for every discrete decision:
argmax best - second similarity, top-r gap s_(r) - s_(r+1), router: the
distance of the count expression to the nearest integer (unclamped only),
exit |c - delta|, prune N (s_(k) - s_(k+1)) for CLS-attention scores
(probabilities of order 1/N) and s_(k) - s_(k+1) for learned scores.

Follow mode: given another implementation's decisions (``follow``), the
oracle checks each against its own and adopts it only when the disagreement
lies inside the decision margin ``tol`` (a near tie, where either choice is
correct); any other disagreement raises ``DecisionMismatch``.  The later
state then continues from the adopted choice, so the comparison never loses
the rest of the sample.

Parity pins live in tests/test_oracle_*.py (plain-ViT library equivalence,
merge invariants, brute force on tiny inputs, exit trajectory, prune sort,
router closed forms).  The merge/prune/router readings themselves are choices
the paper does not fix: parity unpinned beyond those invariants.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf as _erf

F32 = np.float32
TOL = 1e-3

# Accumulation of the matrix products: "fp32" (BLAS sgemm, the default) or
# "fp64" (accumulate in double, round once to float32).  Only the summation
# order differs; the second setting measures how far the bf16 rounding points
# amplify summation-order noise (a property of the arithmetic, not of any
# implementation).
ACCUM = "fp32"


def _mm(a, b):
    if ACCUM == "fp64":
        return (np.asarray(a, np.float64) @ np.asarray(b, np.float64)).astype(F32)
    return a @ b


class accumulate:
    """Context manager selecting ACCUM for the oracle's matrix products."""

    def __init__(self, mode):
        self.mode = mode

    def __enter__(self):
        global ACCUM
        self.prev, ACCUM = ACCUM, self.mode

    def __exit__(self, *exc):
        global ACCUM
        ACCUM = self.prev


class DecisionMismatch(AssertionError):
    pass


# ---------------------------------------------------------------- rounding --
def bf16_round(a):
    """Round float32 values to the nearest bfloat16 (ties to even)."""
    a = np.ascontiguousarray(a, dtype=F32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(F32)


def _rnd(a, mode):
    return bf16_round(a) if mode == "bf16emu" else np.asarray(a, dtype=F32)


# -------------------------------------------------------------- primitives --
def layer_norm(x, g, b, eps=1e-6):
    """LayerNorm over the last axis: biased variance, affine (Eq. 2)."""
    x = np.asarray(x, dtype=F32)
    mu = x.mean(axis=-1, keepdims=True, dtype=F32)
    xc = x - mu
    var = (xc * xc).mean(axis=-1, keepdims=True, dtype=F32)
    return (xc / np.sqrt(var + F32(eps))) * g + b


def gelu(x):
    """Exact GELU, 0.5 x (1 + erf(x / sqrt 2))."""
    x = np.asarray(x, dtype=F32)
    return F32(0.5) * x * (F32(1.0) + _erf(x * F32(1.0 / math.sqrt(2.0))).astype(F32))


def prepare_weights(W: dict, mode: str) -> dict:
    """Round the matrix-product weights once (bf16emu); others stay fp32."""
    out = {}
    for k, v in W.items():
        leaf = k.split(".")[-1]
        if leaf in ("pe_w", "qkv_w", "proj_w", "fc1_w", "fc2_w", "ew", "ew1",
                    "ew2", "head_w"):
            out[k] = _rnd(v, mode)
        else:
            out[k] = np.asarray(v, dtype=F32)
    return out


# ------------------------------------------------------------ patch embed --
def patchify(img, p):
    """[C, H, W] -> [N0, C*p*p]; patches raster order, vectors (c, ky, kx)."""
    C, H, Wd = img.shape
    g = H // p
    t = img.reshape(C, g, p, g, p).transpose(1, 3, 0, 2, 4)
    return np.ascontiguousarray(t.reshape(g * g, C * p * p), dtype=F32)


def patch_embed(img, W, cfg, mode):
    """z_0 = [cls; patches W_pe^T + b_pe] + pos (Eq. 1)."""
    P = _rnd(patchify(img, cfg["patch"]), mode)
    tok = _mm(P, W["pe_w"].T) + W["pe_b"]
    z = np.concatenate([W["cls"][None, :], tok], axis=0)
    return (z + W["pos"]).astype(F32)


# ------------------------------------------------------------------ block --
def attention(x, s, Wb, cfg, mode, want_cls):
    """Multi-head self-attention on LN1(x); returns (O, cls_attn or None).

    q|k|v = round(LN1(x) W_qkv^T + b_qkv), then ``attention_heads``.
    """
    h = _rnd(layer_norm(x, Wb["ln1_g"], Wb["ln1_b"]), mode)
    qkv = _rnd(_mm(h, Wb["qkv_w"].T) + Wb["qkv_b"], mode)
    return attention_heads(qkv, s, cfg["H"], cfg["prop_attn"], mode, want_cls)


def attention_heads(qkv, s, H, prop_attn, mode, want_cls):
    """Multi-head attention of one sample on its q|k|v rows [T, 3d]
    (columns q | k | v, each head-major); returns (O rounded to the storage
    type, cls_attn or None).

    S = (q k^T) * dh^-1/2 + ln(s_key) (proportional attention),
    E = exp(S - rowmax), l = rowsum(E), O = (round(E) V) / l.
    cls_attn[j] = mean over heads of E[0, j] / l[0] (float32, unrounded).
    """
    qkv = np.asarray(qkv, dtype=F32)
    d = qkv.shape[1] // 3
    dh = d // H
    scale = F32(1.0 / math.sqrt(dh))
    bias = np.log(s).astype(F32) if prop_attn else None
    T = qkv.shape[0]
    O = np.empty((T, d), dtype=F32)
    cls_rows = []
    for hh in range(H):
        q = qkv[:, hh * dh:(hh + 1) * dh]
        k = qkv[:, d + hh * dh:d + (hh + 1) * dh]
        v = qkv[:, 2 * d + hh * dh:2 * d + (hh + 1) * dh]
        S = _mm(q, k.T) * scale
        if bias is not None:
            S = S + bias[None, :]
        E = np.exp(S - S.max(axis=1, keepdims=True))
        l = E.sum(axis=1, keepdims=True, dtype=F32)
        O[:, hh * dh:(hh + 1) * dh] = _mm(_rnd(E, mode), v) / l
        if want_cls:
            cls_rows.append(E[0] / l[0])
    cls_attn = None
    if want_cls:
        acc = cls_rows[0].copy()
        for r_ in cls_rows[1:]:
            acc = acc + r_
        cls_attn = (acc / F32(H)).astype(F32)
    return _rnd(O, mode), cls_attn


def block(x, s, Wb, cfg, mode, want_cls=False):
    """Block_b: x += proj(MHSA(LN1 x)); x += fc2(GELU(fc1(LN2 x))) (Eq. 2)."""
    O, cls_attn = attention(x, s, Wb, cfg, mode, want_cls)
    x = x + (_mm(O, Wb["proj_w"].T) + Wb["proj_b"])
    h = _rnd(layer_norm(x, Wb["ln2_g"], Wb["ln2_b"]), mode)
    f = _rnd(gelu(_mm(h, Wb["fc1_w"].T) + Wb["fc1_b"]), mode)
    x = x + (_mm(f, Wb["fc2_w"].T) + Wb["fc2_b"])
    return x.astype(F32), cls_attn


def head_logits(x_cls, g, b, Wh, bh, mode):
    """Linear classifier on LN(CLS) (Eq. 3 and the exit heads of Eq. 6)."""
    y = _rnd(layer_norm(x_cls[None, :], g, b), mode)
    return (_mm(y, Wh.T) + bh)[0].astype(F32)


def mlp_head_logits(v, g, b, W1, b1, W2, b2, mode):
    """2-layer MLP head on a d-vector: LN, W1 + b1, exact GELU, W2 + b2."""
    y = _rnd(layer_norm(v[None, :], g, b), mode)
    h = _rnd(gelu(_mm(y, W1.T) + b1), mode)
    return (_mm(h, W2.T) + b2)[0].astype(F32)


def spatial_pool(x, s):
    """Size-weighted mean of the patch rows: sum_t s_t x_t / sum_t s_t over
    t >= 1, summed in token order; zero vector without patch rows."""
    if x.shape[0] <= 1:
        return np.zeros(x.shape[1], dtype=F32)
    num = np.zeros(x.shape[1], dtype=F32)
    den = F32(0.0)
    for t in range(1, x.shape[0]):
        num = num + s[t] * x[t]
        den = den + s[t]
    return (num / den).astype(F32)


def exit_logits(x, s, Wb, kind, mode):
    """head_b of Eq. 6 for the exit-head kind of the block."""
    if kind == "linear":
        return head_logits(x[0], Wb["eln_g"], Wb["eln_b"], Wb["ew"], Wb["eb"], mode)
    v = x[0] if kind == "cls_mlp" else spatial_pool(x, s)
    return mlp_head_logits(v, Wb["eln_g"], Wb["eln_b"], Wb["ew1"], Wb["eb1"],
                           Wb["ew2"], Wb["eb2"], mode)


def max_softmax(l):
    """c = max_k softmax(l)_k = 1 / sum_k exp(l_k - max l)  (Eq. 7)."""
    e = np.exp(l - l.max())
    return F32(1.0) / e.sum(dtype=F32)


# ------------------------------------------------------------ router ------
def router(x_cls, w, beta, rho, r_b, N, rule="budget"):
    """m = sigmoid(w . z_cls + beta) (Eq. 4); r by the merge-count rule.

    "budget":   r = clamp(floor(2 rho m r_b + 1/2), 0, floor(N/2));
    "fraction": r = min(floor(((rho m) N) / 2), floor(N/2)) (Sec. III-C
                with the rescaled ratio of Eq. 5).
    Returns (m, r, margin).  The margin is the distance of the count
    expression (2 rho m r_b + 1/2, or rho m N / 2) to the nearest integer,
    in units of the count, i.e. how far the expression must move to change
    r; +inf when the count is clamped or does not depend on m.
    """
    z = F32(np.dot(w, x_cls)) + F32(beta)
    m = F32(1.0) / (F32(1.0) + np.exp(-z, dtype=F32))
    if rule == "fraction":
        t = ((float(rho) * float(m)) * float(N)) * 0.5
        slope = 0.5 * float(rho) * float(N)
    else:
        t = ((2.0 * float(rho)) * float(m)) * float(r_b) + 0.5
        slope = 2.0 * float(rho) * float(r_b)
    r_raw = math.floor(t)
    r = min(max(r_raw, 0), N // 2)
    margin = abs(t - round(t)) if (r == r_raw and slope > 0) else math.inf
    return m, int(r), margin


def keep_count(N, tau_b, rho):
    """k = floor(tau' N), tau' = min(1, max(0, 1 - rho (1 - tau_b)))."""
    tau_eff = min(1.0, max(0.0, 1.0 - float(rho) * (1.0 - float(tau_b))))
    return int(math.floor(tau_eff * float(N)))


# ------------------------------------------------------------- merge ------
def merge_plan(x, r):
    """Bipartite soft matching on the patch rows of x (rows 1..N).

    Returns dict with: N, A/B slot lists (patch positions), sim [|A|, |B|],
    best (B index per A), bestsim, chosen (A indices, top r), and margins.
    """
    P = x[1:]
    N = P.shape[0]
    nrm = np.sqrt((P * P).sum(axis=1, dtype=F32))
    xh = P / np.maximum(nrm, F32(1e-12))[:, None]
    A = np.arange(0, N, 2)
    B = np.arange(1, N, 2)
    plan = dict(N=N, A=A, B=B)
    if len(B) == 0 or r == 0:
        plan.update(sim=None, best=None, bestsim=None,
                    chosen=np.zeros(0, dtype=np.int64),
                    argmax_margin=math.inf, topr_margin=math.inf)
        return plan
    sim = (xh[A] @ xh[B].T).astype(F32)
    best = np.argmax(sim, axis=1)             # first max -> lowest B slot
    bestsim = sim[np.arange(len(A)), best]
    order = np.argsort(-bestsim, kind="stable")  # ties -> lowest A slot
    chosen = order[:r]
    if len(B) > 1:
        srt = np.sort(sim[chosen], axis=1)
        am = float((srt[:, -1] - srt[:, -2]).min()) if r > 0 else math.inf
    else:
        am = math.inf
    tm = math.inf
    if 0 < r < len(A):
        tm = float(bestsim[order[r - 1]] - bestsim[order[r]])
    plan.update(sim=sim, best=best, bestsim=bestsim, chosen=chosen,
                argmax_margin=am, topr_margin=tm)
    return plan


def apply_merge(x, s, score, origin, A, B, chosen, dst):
    """Size-weighted merge of A[chosen[i]] into B[dst[i]]; drop the sources.

    x: [T, d]; s, score: [T] (score may be None); origin: [T] ints.
    Sources are added to their destination in ascending A-slot order.
    """
    x = x.copy()
    s = s.copy()
    score = None if score is None else score.copy()
    pairs = sorted(zip((int(c) for c in chosen), (int(t) for t in dst)))
    groups = {}
    for a, b in pairs:
        groups.setdefault(b, []).append(a)
    for b, srcs in groups.items():
        rb = 1 + B[b]
        num = s[rb] * x[rb]
        den = s[rb]
        sc = None if score is None else score[rb]
        for a in srcs:
            ra = 1 + A[a]
            num = num + s[ra] * x[ra]
            den = den + s[ra]
            if sc is not None:
                sc = sc + score[ra]
        x[rb] = num / den
        s[rb] = den
        if score is not None:
            score[rb] = sc
    drop = np.zeros(x.shape[0], dtype=bool)
    for a, _ in pairs:
        drop[1 + A[a]] = True
    keep = ~drop
    return (x[keep], s[keep], None if score is None else score[keep],
            origin[keep])


# ------------------------------------------------------------- prune ------
def learned_scores(x, w, beta):
    """s_i = h_b(z_i) = w . z_i + beta for every row (Eq. 8, linear h_b)."""
    return (_mm(x, w) + F32(beta)).astype(F32)


def prune_plan(score, k, unit=None):
    """Top-k patch tokens by score (ties -> lower position); CLS excluded.

    Returns (kept patch positions in order, margin unit (s_(k) - s_(k+1)),
    order); ``unit`` defaults to N (probability scores of order 1/N).
    """
    sc = score[1:]
    N = sc.shape[0]
    if unit is None:
        unit = float(N)
    order = np.argsort(-sc, kind="stable")
    kept = np.sort(order[:k])
    margin = math.inf
    if 0 < k < N:
        margin = float(unit) * float(sc[order[k - 1]] - sc[order[k]])
    return kept, margin, order


# ----------------------------------------------------------- the sample ---
def _b_weights(W, b):
    p = f"blk{b}."
    return {k[len(p):]: v for k, v in W.items() if k.startswith(p)}


def run_sample(img, W, cfg, mode, delta=None, rho=1.0, follow=None,
               tol=TOL, record=False):
    """Algorithm 1 for one image.  ``W`` must come from ``prepare_weights``.

    delta: exit thresholds per exit block (defaults to cfg["delta"]).
    follow: optional per-block dict {b: {"r": int, "merge": {src_origin:
            dst_origin}, "exit": bool, "ids": [origin ids after the block's
            adaptation]}} from another implementation (see module doc).
    tol:    decision margin under which a followed choice may differ; a
            float, or {"exit": t_exit, "other": t[, "prune": t_prune]
            [, "router": t_router]} to give the exit rule (units of c), the
            prune rule (score units) and the merge count (count units) their
            own margins.
    Returns dict(logits, exit_block, token_counts[L], trace, adopted).
    """
    L = cfg["L"]
    if isinstance(tol, dict):
        tol_exit, tol_prune = tol["exit"], tol.get("prune", tol["other"])
        tol_router, tol = tol.get("router", tol["other"]), tol["other"]
    else:
        tol_exit = tol_prune = tol_router = tol
    if delta is None:
        delta = cfg["delta"]
    delta_of = {b: F32(dl) for b, dl in zip(cfg["exits"], delta)}
    kind_of = dict(zip(cfg["exits"], cfg.get("exit_kind",
                                             ("linear",) * len(cfg["exits"]))))
    merge_rule = cfg.get("merge_rule", "budget")
    learned = cfg.get("prune_rule", "cls_attn") == "learned"
    x = patch_embed(img, W, cfg, mode)
    T0 = x.shape[0]
    s = np.ones(T0, dtype=F32)
    origin = np.arange(T0, dtype=np.int64)
    counts = np.zeros(L, dtype=np.int64)
    trace = {}
    adopted = []
    for b in range(1, L + 1):
        counts[b - 1] = x.shape[0]
        Wb = _b_weights(W, b)
        isM, isE, isP = b in cfg["merges"], b in cfg["exits"], b in cfg["prunes"]
        x, score = block(x, s, Wb, cfg, mode, want_cls=isP and not learned)
        fb = None if follow is None else follow.get(b)
        tb = dict(T=x.shape[0])
        # ---- merge (Alg. 1, merge branch; Sec. III-C)
        if isM:
            N = x.shape[0] - 1
            m, r, rmargin = router(x[0], Wb["router_w"], Wb["router_b"][0],
                                   rho, cfg["r_b"][b - 1], N, merge_rule)
            tb.update(m=float(m), r=r, router_margin=rmargin)
            if fb is not None and fb["r"] != r:
                if not (rmargin < tol_router and abs(fb["r"] - r) == 1):
                    raise DecisionMismatch(
                        f"block {b}: r {fb['r']} vs oracle {r} (margin {rmargin})")
                adopted.append((b, "r"))
                r = fb["r"]
            plan = merge_plan(x, r)
            chosen, dst = plan["chosen"], (None if r == 0 else plan["best"][plan["chosen"]])
            if fb is not None:
                chosen, dst = _follow_merge(b, plan, r, origin, fb["merge"], tol,
                                            adopted)
            tb.update(argmax_margin=plan["argmax_margin"],
                      topr_margin=plan["topr_margin"])
            mmap = {}
            for a, t in zip(chosen, dst if dst is not None else []):
                mmap[int(origin[1 + plan["A"][a]])] = int(origin[1 + plan["B"][t]])
            tb["merge"] = mmap
            if r > 0:
                x, s, score, origin = apply_merge(x, s, score, origin,
                                                  plan["A"], plan["B"],
                                                  chosen, dst)
            tb["ids_after_merge"] = origin.copy()
        # ---- exit check (Alg. 1, exit branch; Sec. III-D)
        if isE:
            lg = exit_logits(x, s, Wb, kind_of[b], mode)
            c = max_softmax(lg)
            dl = delta_of[b]
            fire = bool(dl < F32(1.0) and c >= dl)
            tb.update(c=float(c), exit_margin=abs(float(c) - float(dl)),
                      exit_logits=lg)
            if fb is not None and fb["exit"] != fire:
                if not abs(float(c) - float(dl)) < tol_exit:
                    raise DecisionMismatch(f"block {b}: exit {fb['exit']} vs oracle {fire} (c={c}, delta={dl})")
                adopted.append((b, "exit"))
                fire = fb["exit"]
            tb["exit"] = fire
            if fire:
                trace[b] = tb
                return dict(logits=lg, exit_block=b, token_counts=counts,
                            trace=trace, adopted=adopted)
        # ---- prune, continuing samples only (Alg. 1, prune branch; Sec. III-E)
        if isP:
            N = x.shape[0] - 1
            k = keep_count(N, cfg["tau_b"][b - 1], rho)
            unit = None
            if learned:
                score = learned_scores(x, Wb["prune_w"], Wb["prune_b"][0])
                unit = 1.0
            kept, pmargin, order = prune_plan(score, k, unit)
            tb.update(k=k, prune_margin=pmargin, scores=score.copy(),
                      score_unit=1.0 if learned else float(N))
            if fb is not None:
                kept = _follow_prune(b, score, k, kept, order, origin, fb["ids"],
                                     tol_prune, adopted, unit)
            rows = np.concatenate([[0], 1 + kept]).astype(np.int64)
            x, s, origin = x[rows], s[rows], origin[rows]
        tb["ids"] = origin.copy()
        if fb is not None and not np.array_equal(np.asarray(fb["ids"]), origin):
            raise DecisionMismatch(f"block {b}: surviving ids differ")
        trace[b] = tb
    lg = head_logits(x[0], W["norm_g"], W["norm_b"], W["head_w"], W["head_b"], mode)
    return dict(logits=lg, exit_block=L, token_counts=counts, trace=trace,
                adopted=adopted)


def _follow_merge(b, plan, r, origin, fmerge, tol, adopted):
    """Check another implementation's merge map against the oracle's plan."""
    A, B = plan["A"], plan["B"]
    if len(fmerge) != r:
        raise DecisionMismatch(f"block {b}: {len(fmerge)} merges vs r={r}")
    if r == 0:
        return plan["chosen"], None
    a_of = {int(origin[1 + a]): i for i, a in enumerate(A)}
    b_of = {int(origin[1 + t]): i for i, t in enumerate(B)}
    chosen_f, dst_f = [], []
    for so, do in fmerge.items():
        if so not in a_of or do not in b_of:
            raise DecisionMismatch(f"block {b}: merge {so}->{do} not an A->B pair")
        chosen_f.append(a_of[so])
        dst_f.append(b_of[do])
    chosen_f = np.array(chosen_f)
    dst_f = np.array(dst_f)
    bs = plan["bestsim"]
    order = np.argsort(-bs, kind="stable")
    s_r = bs[order[r - 1]]
    s_r1 = bs[order[r]] if r < len(A) else -np.inf
    own = set(int(c) for c in plan["chosen"])
    theirs = set(int(c) for c in chosen_f)
    for a in theirs - own:
        if not bs[a] >= s_r - tol:
            raise DecisionMismatch(f"block {b}: chose A{a} (sim {bs[a]}) vs s_r {s_r}")
    for a in own - theirs:
        if not bs[a] <= s_r1 + tol:
            raise DecisionMismatch(f"block {b}: skipped A{a} (sim {bs[a]}) vs s_r+1 {s_r1}")
    if own != theirs:
        adopted.append((b, "topr"))
    for a, t in zip(chosen_f, dst_f):
        if t != plan["best"][a]:
            if not plan["sim"][a, t] >= bs[a] - tol:
                raise DecisionMismatch(f"block {b}: A{a}->B{t} sim {plan['sim'][a, t]} vs best {bs[a]}")
            adopted.append((b, "argmax"))
    return chosen_f, dst_f


def _follow_prune(b, score, k, kept, order, origin, fids, tol, adopted,
                  unit=None):
    sc = score[1:]
    N = sc.shape[0]
    U = float(N) if unit is None else float(unit)
    pos_of = {int(o): i for i, o in enumerate(origin[1:])}
    fids = [int(t) for t in fids]
    if len(fids) != k + 1 or fids[0] != int(origin[0]):
        raise DecisionMismatch(f"block {b}: kept {len(fids) - 1} vs k={k}")
    theirs = set()
    for o in fids[1:]:
        if o not in pos_of:
            raise DecisionMismatch(f"block {b}: kept unknown token {o}")
        theirs.add(pos_of[o])
    own = set(int(t) for t in kept)
    if own == theirs:
        return kept
    s_k = sc[order[k - 1]] if k > 0 else np.inf
    s_k1 = sc[order[k]] if k < N else -np.inf
    for t in theirs - own:
        if not U * sc[t] >= U * s_k - tol:
            raise DecisionMismatch(f"block {b}: kept pos {t} score {sc[t]} vs s_k {s_k}")
    for t in own - theirs:
        if not U * sc[t] <= U * s_k1 + tol:
            raise DecisionMismatch(f"block {b}: pruned pos {t} score {sc[t]} vs s_k+1 {s_k1}")
    adopted.append((b, "prune"))
    return np.array(sorted(theirs), dtype=np.int64)


def run(images, W_raw, cfg, mode, delta=None, rho=1.0, follow=None, tol=TOL):
    """Run every image; returns logits [B, C], exit_block [B], counts [B, L],
    and the per-sample results list."""
    W = prepare_weights(W_raw, mode)
    res = []
    for i in range(images.shape[0]):
        f = None if follow is None else follow[i]
        res.append(run_sample(images[i], W, cfg, mode, delta, rho, f, tol))
    logits = np.stack([r_["logits"] for r_ in res])
    exit_block = np.array([r_["exit_block"] for r_ in res], dtype=np.int64)
    counts = np.stack([r_["token_counts"] for r_ in res])
    return logits, exit_block, counts, res


def plain_forward(img, W, cfg, mode):
    """The unadapted ViT: patch embed, L blocks with unit sizes, final head."""
    x = patch_embed(img, W, cfg, mode)
    s = np.ones(x.shape[0], dtype=F32)
    for b in range(1, cfg["L"] + 1):
        x, _ = block(x, s, _b_weights(W, b), cfg, mode)
    return head_logits(x[0], W["norm_g"], W["norm_b"], W["head_w"],
                       W["head_b"], mode)


def executed_flops(cfg, token_counts, exit_block):
    """Algorithmic FLOPs actually executed for one sample.

    Per executed block with T tokens: 24 T d^2 (+ 8 T d mlp/d correction
    for mlp != 4d) + 4 T^2 d; patch embed 2 N0 (C p^2) d; per head
    evaluated (exit heads reached, final head if no exit) 2 d C for a
    linear head and 2 d h + 2 h C for an MLP head of hidden width h.  Only
    matrix products count (no LayerNorm, pooling, softmax or scorer).
    """
    d, mlp, C = cfg["d"], cfg["mlp"], cfg["C"]
    kinds = dict(zip(cfg["exits"], cfg.get("exit_kind",
                                           ("linear",) * len(cfg["exits"]))))
    hx = cfg.get("exit_hidden", 0)
    f = 2 * cfg["N0"] * cfg["patch_dim"] * d
    for b in range(1, cfg["L"] + 1):
        T = int(token_counts[b - 1])
        if T == 0:
            continue
        f += 2 * T * d * 3 * d + 2 * T * d * d + 4 * T * d * mlp + 4 * T * T * d
        if b in cfg["exits"]:
            f += 2 * d * C if kinds[b] == "linear" else 2 * d * hx + 2 * hx * C
    if exit_block == cfg["L"]:
        f += 2 * d * C
    return f
