"""fp64 CPU oracle for verifier-side window scoring (Interactive-Policy Distillation).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import or call this module.  It shares no
code with the HIP library or its Python binding and imports neither.

What it computes, each part written from the paper's definitions:

* ``verify_attn_paged`` -- the verification stage of one fused-engine step
  (Section 3.2.3, "Fused Inference Engine"): the verifier appends the window's
  keys/values to its own paged cache and scores every window row in one
  prefill pass over the resident prefix.  Plain causal softmax attention,
  evaluated per row and head in fp64.
* ``lmhead_logsoftmax`` -- the verifier's next-token distribution at each
  window row: logits, their log-softmax (temperature 1, Appendix A), the
  proposed token's log-prob (the log q / log pi term of Eq. (4)), the top-K
  support of Eq. (5) and the entropy.  Top-K is a full stable sort by
  (logit descending, index ascending).
* ``accept_scan`` -- the verdict stage (Section 3.2.3) applying the top-K
  coverage transition of Eq. (9) over a window with the EOS and maximum
  length rules, and the rule variants named after Eq. (9) in Section 3.2.1
  (entropy thresholds, asymmetric rules, SKD's fixed one-token handback);
  ``eq9_stepper`` is a second, token-by-token writing of Eq. (9) used to
  cross-check it.
* ``sample_takeover`` -- the teacher's replacement token at a takeover
  (Eq. (9), second case: the uncovered student draft is discarded and the
  teacher samples a replacement from its own distribution at that position,
  temperature 1), drawn by inverse CDF over the vocabulary in index order
  from a caller-supplied uniform.
* ``source_split_kl`` -- the per-position values of the source-split
  objective (Section 3.2.2): both models renormalised on the top-K support
  (Eqs. (5), (6)), reverse KL at student-generated positions and forward KL
  at teacher-generated ones (Eq. (10)), the length-normalised sum per
  trajectory (Eq. (11)), the top-K overlap ratio and the intervention ratio;
  ``logp_gather`` gives each model's log-probs at the other's top-K indices.
* ``propose_decode`` -- the driver's gamma autoregressive draft steps over
  its own paged cache (Section 3.2.3, propose stage): a one-row attention
  window, the LM head and a temperature-1 draw per step.

Readings where the paper is silent (tie-break, window/row alignment, cache
rollback lengths, EOS inside a window, length cap) are listed in the
repository's design notes; each is restated at the function that uses it.

Cache layouts (the library's documented layouts):
``k_cache[num_pages, Hkv, D/32, page_size, 32]`` -- key channel d of a slot is
at [.., d // 32, slot, d % 32] -- and ``v_cache[num_pages, Hkv, D, page_size]``.
"""
from __future__ import annotations

import numpy as np

DRIVER_S = 0          # the student drives; the teacher verifies
DRIVER_T = 1          # the teacher drives; the student verifies
SRC_S = 0             # token emitted from the student's proposal
SRC_T = 1             # token emitted from the teacher's proposal
SRC_DISCARDED = 255   # draft not emitted


def _f64(x):
    """Exact upcast of an input array (fp32 / bf16-valued) to fp64."""
    return np.asarray(x, dtype=np.float64)


def _seq_list(n_seq, seq_ids):
    return list(range(n_seq)) if seq_ids is None else [int(s) for s in seq_ids]


# ---------------------------------------------------------------------------
# Verification stage: append + causal attention over the paged cache
# ---------------------------------------------------------------------------

def append_window(k_cache, v_cache, k_new, v_new, page_table, ctx_lens, cu_q,
                  seq_ids=None, n_seq=None):
    """Write each window row's key/value into the verifier's pages (in place).

    Row i of sequence b is the token at absolute position L_b + i; it goes to
    page ``page_table[b][(L_b+i) // ps]``, slot ``(L_b+i) % ps`` -- appending
    externally proposed tokens to a live request's cache (Section 3.2.3).
    """
    Hkv, nslice, ps, x = k_cache.shape[1:]
    n_seq = len(ctx_lens) if n_seq is None else n_seq
    for b in _seq_list(n_seq, seq_ids):
        L = int(ctx_lens[b])
        for i in range(int(cu_q[b + 1]) - int(cu_q[b])):
            row = int(cu_q[b]) + i
            pos = L + i
            page = int(page_table[b][pos // ps])
            k_cache[page, :, :, pos % ps, :] = np.reshape(k_new[row], (Hkv, nslice, x))
            v_cache[page, :, :, pos % ps] = v_new[row]


def gather_sequence(k_cache, v_cache, page_table, b, n_tokens):
    """Keys and values of positions [0, n_tokens) of sequence b, as fp64
    arrays [n_tokens, Hkv, D]."""
    Hkv, nslice, ps, x = k_cache.shape[1:]
    pos = np.arange(n_tokens)
    pages = np.asarray(page_table[b])[pos // ps].astype(np.int64)
    slots = pos % ps
    K = _f64(k_cache[pages, :, :, slots, :]).reshape(n_tokens, Hkv, nslice * x)   # [n, Hkv, D]
    V = _f64(v_cache[pages, :, :, slots])                                           # [n, Hkv, D]
    return K, V


def attention_rows(q, K, V, L, scale, Hkv):
    """Causal attention of k window rows q[k, Hq, D] whose keys are K/V[L+k, Hkv, D].

    Row i sees keys 0 .. L+i inclusive.  Query head h reads KV head
    h // (Hq/Hkv) (contiguous grouped-query groups).  Softmax is
    exp(s - max s) / sum, evaluated in fp64.
    """
    q = _f64(q)
    k_rows, Hq, D = q.shape
    group = Hq // Hkv
    out = np.zeros((k_rows, Hq, D), np.float64)
    for i in range(k_rows):
        n_vis = L + i + 1
        for h in range(Hq):
            g = h // group
            s = (K[:n_vis, g, :] @ q[i, h, :]) * scale
            p = np.exp(s - s.max())
            p /= p.sum()
            out[i, h, :] = p @ V[:n_vis, g, :]
    return out


def verify_attention(q, k_cache, v_cache, page_table, ctx_lens, cu_q, scale,
                     seq_ids=None, n_seq=None, out=None):
    """Attention of every window row over its sequence's cache, which must
    already hold the window (see ``append_window``).  Returns fp64 [T, Hq, D];
    rows of sequences not in ``seq_ids`` are left as in ``out`` (zeros)."""
    T, Hq, D = q.shape
    Hkv = k_cache.shape[1]
    n_seq = len(ctx_lens) if n_seq is None else n_seq
    if out is None:
        out = np.zeros((T, Hq, D), np.float64)
    for b in _seq_list(n_seq, seq_ids):
        L = int(ctx_lens[b])
        r0, r1 = int(cu_q[b]), int(cu_q[b + 1])
        if r1 == r0:
            continue
        K, V = gather_sequence(k_cache, v_cache, page_table, b, L + (r1 - r0))
        out[r0:r1] = attention_rows(q[r0:r1], K, V, L, scale, Hkv)
    return out


def verify_attn_paged(q, k_new, v_new, k_cache, v_cache, page_table, ctx_lens, cu_q,
                      scale, seq_ids=None, n_seq=None):
    """The whole verification-stage attention: append the window to copies of
    the caches, then attend.  Returns (out fp64 [T,Hq,D], k_cache', v_cache')."""
    kc = np.array(k_cache, copy=True)
    vc = np.array(v_cache, copy=True)
    append_window(kc, vc, k_new, v_new, page_table, ctx_lens, cu_q, seq_ids, n_seq)
    out = verify_attention(q, kc, vc, page_table, ctx_lens, cu_q, scale, seq_ids, n_seq)
    return out, kc, vc


# ---------------------------------------------------------------------------
# LM head + vocabulary log-softmax + top-K support
# ---------------------------------------------------------------------------

def logits_fp64(hidden, W, chunk=16384):
    """l = h W^T in fp64, [M, V] (W is [V, Hd], the nn.Linear layout)."""
    h = _f64(hidden)
    V = W.shape[0]
    out = np.empty((h.shape[0], V), np.float64)
    for v0 in range(0, V, chunk):
        out[:, v0:v0 + chunk] = h @ _f64(W[v0:v0 + chunk]).T
    return out


def lmhead_logsoftmax(hidden, W, prop_tok, K, logits=None):
    """Verifier outputs for each row: log-softmax, proposal log-prob, top-K.

    Top-K (Eq. (5)) is the first K entries of a stable sort of the row by
    logit descending, so equal logits keep ascending index order (the paper
    does not fix the tie-break; lower index wins here).  Argmax is the first
    entry of that order.  Entropy is -sum_v p_v log p_v.

    Also returns the decision margins used by parity checks:
    ``argmax_margin`` = l_(1) - l_(2); ``set_margin`` = l_(K) - l_(K+1);
    ``cover_margin`` = l_prop - l_(K+1) if the proposal is in the top-K,
    else l_(K) - l_prop (inf where undefined).
    """
    l = logits_fp64(hidden, W) if logits is None else _f64(logits)
    M, V = l.shape
    Kc = min(int(K), V)
    mx = l.max(axis=1)
    lse = mx + np.log(np.exp(l - mx[:, None]).sum(axis=1))
    logp = l - lse[:, None]
    prop = np.asarray(prop_tok, np.int64)
    res = {
        "lse": lse,
        "logp_prop": logp[np.arange(M), prop],
        "argmax": np.zeros(M, np.int64),
        "topk_idx": np.zeros((M, Kc), np.int64),
        "topk_logp": np.zeros((M, Kc), np.float64),
        "entropy": -(np.exp(logp) * logp).sum(axis=1),
        "argmax_margin": np.full(M, np.inf),
        "set_margin": np.full(M, np.inf),
        "cover_margin": np.full(M, np.inf),
        "covered": np.zeros(M, bool),
    }
    for m in range(M):
        order = np.argsort(-l[m], kind="stable")
        res["argmax"][m] = order[0]
        res["topk_idx"][m] = order[:Kc]
        res["topk_logp"][m] = logp[m, order[:Kc]]
        if V > 1:
            res["argmax_margin"][m] = l[m, order[0]] - l[m, order[1]]
        rank = int(np.nonzero(order == prop[m])[0][0])
        res["covered"][m] = rank < Kc
        if 0 < Kc < V:
            res["set_margin"][m] = l[m, order[Kc - 1]] - l[m, order[Kc]]
            if rank < Kc:
                res["cover_margin"][m] = l[m, prop[m]] - l[m, order[Kc]]
            else:
                res["cover_margin"][m] = l[m, order[Kc - 1]] - l[m, prop[m]]
    return res


# ---------------------------------------------------------------------------
# Verdict stage: top-K coverage rule of Eq. (9) over a window
# ---------------------------------------------------------------------------

# Takeover and handback rules (Section 3.2.1, after Eq. (9): the coverage
# rules are the paper's default; an entropy threshold can replace either, the
# two may differ, and SKD is coverage takeover with a fixed one-token handback).
TAKE_COVERAGE = 0     # take over when the student's draft is outside the teacher's top-K
TAKE_ENTROPY = 1      # take over when ent[row] > tau_take
HAND_COVERAGE = 0     # hand back when the teacher's draft is inside the student's top-K
HAND_FIXED_ONE = 1    # the teacher emits one token, then hands back (SKD)
HAND_ENTROPY = 2      # hand back when ent[row] <= tau_hand


def _rule_tests(row, tok, topk_row, K, take_rule, hand_rule, ent, tau_take, tau_hand):
    """(takeover test, handback test) for one window row.

    Coverage: the draft is among the verifier's K entries.  Entropy: a
    threshold on the caller's per-row entropy (which model's entropy it is --
    the paper allows either -- is the caller's choice); a NaN entropy passes
    neither test.  Fixed one-token handback: every teacher token hands back.
    """
    covered = K > 0 and tok in [int(t) for t in topk_row[:K]]
    if take_rule == TAKE_COVERAGE:
        take = not covered
    elif take_rule == TAKE_ENTROPY:
        take = bool(float(ent[row]) > tau_take)
    else:
        raise ValueError("unknown takeover rule")
    if hand_rule == HAND_COVERAGE:
        hand = covered
    elif hand_rule == HAND_FIXED_ONE:
        hand = True
    elif hand_rule == HAND_ENTROPY:
        hand = bool(float(ent[row]) <= tau_hand)
    else:
        raise ValueError("unknown handback rule")
    return take, hand


def accept_scan(cu_q, prop_tok, topk_idx, K, driver, ctx_lens, seq_lens, eos_id, max_len,
                take_rule=TAKE_COVERAGE, hand_rule=HAND_COVERAGE, ent=None,
                tau_take=0.0, tau_hand=0.0):
    """Verdict for every sequence's window (Eq. (9), Section 3.2.3).

    Row i of sequence b scores draft i (``prop_tok[cu_q[b]+i]``), proposed by
    the driver.  With the default rules, take_i = the draft is not in the
    verifier's top-K at that row and hand_i = it is (top-K coverage).

    * Driver S (teacher verifies): drafts are accepted (source S) until the
      first row with take_i.  That row is a takeover: the draft is rejected,
      the teacher will emit a replacement there (sampled later), and the next
      driver is T -- or S under the fixed one-token handback, where the
      replacement is the teacher's only token (SKD, Section 2).
    * Driver T (student verifies): drafts are accepted (source T).  The first
      row with hand_i is a handback: it is kept, later drafts are discarded and
      the next driver is S.
    * EOS: a student EOS ends the request only if it passes the takeover test
      (else takeover); a teacher EOS is accepted and ends it.  Drafts after it
      are discarded.
    * Length cap: draft i needs seq_len + i < max_len; a request whose
      accepted drafts reach max_len ends (a takeover's replacement is checked
      by the caller when it is sampled).

    Rule variants (Section 3.2.1, after Eq. (9)): ``take_rule`` and
    ``hand_rule`` pick the tests independently (asymmetric rules), with
    ``ent[row]`` and the thresholds for the entropy rules.

    Returns arrays: n_acc, event_row (-1: no transition), next_driver,
    finished, new_cache_len, and src[T] (0 S, 1 T, 255 discarded).
    new_cache_len = L_b + n_acc, plus one after a takeover (the rejected
    row's input token stays cached; the replacement becomes the last token).
    """
    cu_q = np.asarray(cu_q, np.int64)
    B = len(cu_q) - 1
    T = int(cu_q[-1])
    if (take_rule == TAKE_ENTROPY or hand_rule == HAND_ENTROPY) and ent is None:
        raise ValueError("an entropy rule needs ent")
    n_acc = np.zeros(B, np.int64)
    event_row = np.full(B, -1, np.int64)
    next_driver = np.asarray(driver, np.int64).copy()
    finished = np.zeros(B, np.int64)
    new_cache_len = np.zeros(B, np.int64)
    src = np.full(T, SRC_DISCARDED, np.int64)
    for b in range(B):
        r0, r1 = int(cu_q[b]), int(cu_q[b + 1])
        drv = int(driver[b])
        takeover = False
        for i in range(r1 - r0):
            row = r0 + i
            if int(seq_lens[b]) + i >= int(max_len):
                finished[b] = 1
                break
            tok = int(prop_tok[row])
            take, hand = _rule_tests(row, tok, topk_idx[row], K, take_rule, hand_rule, ent,
                                     tau_take, tau_hand)
            if drv == DRIVER_S:
                if take:
                    event_row[b] = i
                    next_driver[b] = DRIVER_S if hand_rule == HAND_FIXED_ONE else DRIVER_T
                    takeover = True
                    break
                src[row] = SRC_S
                n_acc[b] = i + 1
                stop = tok == eos_id
            else:
                src[row] = SRC_T
                n_acc[b] = i + 1
                if hand:
                    event_row[b] = i
                    next_driver[b] = DRIVER_S
                stop = hand or tok == eos_id
            if tok == eos_id or int(seq_lens[b]) + n_acc[b] >= int(max_len):
                finished[b] = 1
                stop = True
            if stop:
                break
        new_cache_len[b] = int(ctx_lens[b]) + n_acc[b] + (1 if takeover else 0)
    return {"n_acc": n_acc, "event_row": event_row, "next_driver": next_driver,
            "finished": finished, "new_cache_len": new_cache_len, "src": src}


REPLACEMENT = -1   # placeholder for the teacher's replacement token


def eq9_stepper(drafts, verifier_topk, K, m1, eos_id, room, take_rule=TAKE_COVERAGE,
                hand_rule=HAND_COVERAGE, ent=None, tau_take=0.0, tau_hand=0.0):
    """Token-by-token iteration of Eq. (9) over one window (second writing).

    ``drafts[t]`` is the driver's proposal at step t and ``verifier_topk[t]``
    the verifier's support S_t.  Each step emits (x_t, z_t) and sets m_{t+1}
    by the four cases of Eq. (9).  The remaining drafts were proposed by the
    old driver, so the walk stops as soon as the driver changes, at an
    emitted EOS, or when ``room`` tokens have been emitted.  A takeover emits
    the placeholder REPLACEMENT (the teacher samples it later).

    Rule variants (Section 3.2.1, after Eq. (9)): case 2 fires on the
    takeover test and case 3 on the handback test of ``take_rule`` /
    ``hand_rule`` (coverage by default; ``ent[t]`` for the entropy rules).
    Under the fixed one-token handback (SKD), the teacher's replacement is its
    only token: case 2 then hands control straight back (m_{t+1} = S), and a
    teacher-driven step always takes case 3.

    Returns (emitted tokens, their sources, final driver, finished flag).
    """
    m = m1
    xs, zs = [], []
    finished = False
    for t, x_tilde in enumerate(drafts):
        if len(xs) >= room:
            finished = True
            break
        in_support = x_tilde in list(verifier_topk[t])[:K] if K > 0 else False
        if take_rule == TAKE_COVERAGE:
            take = not in_support
        else:
            take = ent[t] > tau_take
        if hand_rule == HAND_COVERAGE:
            hand = in_support
        elif hand_rule == HAND_FIXED_ONE:
            hand = True
        else:
            hand = ent[t] <= tau_hand
        if m == DRIVER_S and not take:             # case 1
            x, z, m_next = x_tilde, SRC_S, DRIVER_S
        elif m == DRIVER_S:                        # case 2: takeover
            x, z = REPLACEMENT, SRC_T
            m_next = DRIVER_S if hand_rule == HAND_FIXED_ONE else DRIVER_T
        elif hand:                                 # case 3: handback
            x, z, m_next = x_tilde, SRC_T, DRIVER_S
        else:                                      # case 4
            x, z, m_next = x_tilde, SRC_T, DRIVER_T
        xs.append(x)
        zs.append(z)
        changed = m_next != m or x == REPLACEMENT
        m = m_next
        if x == eos_id or (x != REPLACEMENT and len(xs) >= room):
            finished = True
            break
        if changed:
            break
    return xs, zs, m, finished


# ---------------------------------------------------------------------------
# Takeover replacement: a draw from the teacher's distribution
# ---------------------------------------------------------------------------

def sample_categorical(logits, u):
    """Inverse-CDF draw from softmax(logits) at temperature 1 (the rollout
    temperature of the paper's setup) with the uniform u in [0, 1): the first
    vocabulary index v (index order) whose cumulative probability exceeds u.

    Returns (token, margin): margin is the distance of u from the nearer end
    of the token's cumulative-probability interval [C(v-1), C(v)); a draw whose
    margin exceeds the numerical error of a computation is the same in any
    correct implementation of this definition."""
    l = _f64(logits)
    p = np.exp(l - l.max())
    p /= p.sum()
    c = np.cumsum(p)
    v = int(np.searchsorted(c, u, side="right"))     # first index with c[v] > u
    v = min(v, len(l) - 1)
    lo = c[v - 1] if v > 0 else 0.0
    return v, float(min(u - lo, c[v] - u))


def sample_takeover(cu_q, driver, event_row, logits, u, eos_id):
    """Replacement tokens for the takeovers of one verify step (Eq. (9),
    second case; Section 3.2.3: the rejected student token is regenerated by
    the teacher).  A sequence driven by the student (teacher verifying) whose
    window has an event at row j -- necessarily a takeover -- gets
    sample_categorical(logits[cu_q[b] + j], u[b]); the step is finished when
    that token is EOS (a teacher-generated EOS is accepted directly).  Every
    other sequence gets -1.

    Returns a dict with ``token [B]``, ``eos [B]`` (bool) and ``margin [B]``
    (inf where nothing is drawn)."""
    B = len(driver)
    token = np.full(B, -1, dtype=np.int64)
    eos = np.zeros(B, dtype=bool)
    margin = np.full(B, np.inf)
    for b in range(B):
        if int(driver[b]) != DRIVER_S or int(event_row[b]) < 0:
            continue
        r = int(cu_q[b]) + int(event_row[b])
        token[b], margin[b] = sample_categorical(logits[r], float(u[b]))
        eos[b] = token[b] == eos_id
    return {"token": token, "eos": eos, "margin": margin}


# ---------------------------------------------------------------------------
# Source-split KL values on the top-K support (Eqs. (5), (6), (10), (11))
# ---------------------------------------------------------------------------

# Distillation support S_t (Eq. (5) and the text after it; Appendix B.2: the
# union is the paper's default).
SUPPORT_UNION = 0
SUPPORT_STUDENT = 1
SUPPORT_TEACHER = 2
SUPPORT_INTERSECTION = 3
# KL direction per token source (Eq. (10) is the default; Section 4.3 ablates
# the other three).
LOSS_IPD_SPLIT = 0       # reverse KL where z = S, forward KL where z = T
LOSS_PURE_REVERSE = 1
LOSS_PURE_FORWARD = 2
LOSS_INVERSE_SPLIT = 3   # forward KL where z = S, reverse KL where z = T


def logp_gather(hidden, W, idx, logits=None):
    """log-softmax of the row's logits at the given vocabulary indices.

    ``idx [M, n]``; entries outside [0, V) give -inf.  Each model's log-probs
    at the other model's top-K indices complete the union support of Eq. (6).
    """
    l = logits_fp64(hidden, W) if logits is None else _f64(logits)
    M, V = l.shape
    mx = l.max(axis=1)
    lse = mx + np.log(np.exp(l - mx[:, None]).sum(axis=1))
    idx = np.asarray(idx, np.int64)
    out = np.full(idx.shape, -np.inf)
    for m in range(M):
        for j, v in enumerate(idx[m]):
            if 0 <= v < V:
                out[m, j] = l[m, v] - lse[m]
    return out


def _topk_set(logp_row, K):
    """Top_K of Eq. (5): the first K of a stable sort by log-prob descending
    (equal values: lower index first)."""
    return [int(v) for v in np.argsort(-logp_row, kind="stable")[:K]]


def _support(Sp, Sq, support):
    if support == SUPPORT_UNION:
        return Sp + [v for v in Sq if v not in Sp]
    if support == SUPPORT_STUDENT:
        return list(Sp)
    if support == SUPPORT_TEACHER:
        return list(Sq)
    if support == SUPPORT_INTERSECTION:
        return [v for v in Sp if v in Sq]
    raise ValueError("unknown support")


def _kl_pair(lp, lq):
    """(D(pi_bar || q_bar), D(q_bar || pi_bar)) of Eq. (6)'s renormalised
    distributions from log-probs on the support; an empty support gives 0."""
    lp = np.asarray(lp, np.float64)
    lq = np.asarray(lq, np.float64)
    if lp.size == 0:
        return 0.0, 0.0
    a = lp - (lp.max() + np.log(np.exp(lp - lp.max()).sum()))   # log pi_bar
    b = lq - (lq.max() + np.log(np.exp(lq - lq.max()).sum()))   # log q_bar
    rev = float((np.exp(a) * (a - b)).sum())
    fwd = float((np.exp(b) * (b - a)).sum())
    return rev, fwd


def _row_loss(rev, fwd, z, loss_mode):
    if z == SRC_DISCARDED:
        return 0.0
    on = z == SRC_S
    if loss_mode == LOSS_IPD_SPLIT:
        return rev if on else fwd
    if loss_mode == LOSS_PURE_REVERSE:
        return rev
    if loss_mode == LOSS_PURE_FORWARD:
        return fwd
    if loss_mode == LOSS_INVERSE_SPLIT:
        return fwd if on else rev
    raise ValueError("unknown loss mode")


def _segments(rows_loss, src, cu):
    """Eq. (11)'s inner term per trajectory segment: the mean of the row losses
    over the emitted tokens (src S or T), and the teacher-intervention ratio
    (the share of teacher-generated tokens, Section 4.3).  A segment with no
    emitted token gives 0 for both."""
    cu = np.asarray(cu, np.int64)
    B = len(cu) - 1
    seq_loss = np.zeros(B)
    t_ratio = np.zeros(B)
    for b in range(B):
        z = np.asarray(src[cu[b]:cu[b + 1]])
        keep = z != SRC_DISCARDED
        n = int(keep.sum())
        if n:
            seq_loss[b] = float(np.asarray(rows_loss[cu[b]:cu[b + 1]])[keep].sum()) / n
            t_ratio[b] = float((z == SRC_T).sum()) / n
    return seq_loss, t_ratio


def source_split_kl(logp_student, logp_teacher, K, src, support=SUPPORT_UNION,
                    loss_mode=LOSS_IPD_SPLIT, cu=None):
    """Per-position source-split KL values (Section 3.2.2).

    ``logp_student`` / ``logp_teacher`` ``[M, V]`` are the two models' full
    log-softmax at the same positions c_t; ``src [M]`` the token sources z_t.
    Per row: S^pi and S^q (Eq. (5)), the support S_t, both distributions
    renormalised on it (Eq. (6)), the reverse KL D(pi_bar || q_bar) and the
    forward KL D(q_bar || pi_bar) (Eq. (10)), the row's loss by source
    (``loss_mode``; discarded rows give 0) and the top-K overlap ratio
    |S^pi n S^q| / K (Section 4.2).  With ``cu`` (segment offsets, one
    segment per trajectory) also the length-normalised loss of Eq. (11) and
    the intervention ratio per segment.
    """
    lps = _f64(logp_student)
    lpt = _f64(logp_teacher)
    M = lps.shape[0]
    out = {k: np.zeros(M) for k in ("kl_rev", "kl_fwd", "loss", "overlap")}
    for m in range(M):
        Sp = _topk_set(lps[m], K)
        Sq = _topk_set(lpt[m], K)
        S = _support(Sp, Sq, support)
        rev, fwd = _kl_pair(lps[m, S], lpt[m, S])
        out["kl_rev"][m], out["kl_fwd"][m] = rev, fwd
        out["loss"][m] = _row_loss(rev, fwd, int(src[m]), loss_mode)
        out["overlap"][m] = len(set(Sp) & set(Sq)) / K
    if cu is not None:
        out["seq_loss"], out["t_ratio"] = _segments(out["loss"], src, cu)
    return out


def source_split_kl_lists(s_idx, s_logp, s_at_t, t_idx, t_logp, t_at_s, src,
                          support=SUPPORT_UNION, loss_mode=LOSS_IPD_SPLIT, cu=None):
    """``source_split_kl`` from what the verifier path produces instead of
    full log-prob rows: each model's top-K indices and log-probs
    (``s_idx, s_logp``; ``t_idx, t_logp``, each ``[M, K]``) and each model's
    log-probs at the other's top-K indices (``s_at_t`` = student at t_idx,
    ``t_at_s`` = teacher at s_idx).

    An index in both lists takes its two log-probs from the list that defines
    the support: the student's list (s_logp, t_at_s) for the union, S^pi and
    the intersection; the teacher's (s_at_t, t_logp) for S^q.
    """
    s_idx = np.asarray(s_idx, np.int64)
    t_idx = np.asarray(t_idx, np.int64)
    M, K = s_idx.shape
    out = {k: np.zeros(M) for k in ("kl_rev", "kl_fwd", "loss", "overlap")}
    for m in range(M):
        Sp, Sq = list(s_idx[m]), list(t_idx[m])
        lp, lq = [], []
        if support in (SUPPORT_UNION, SUPPORT_STUDENT, SUPPORT_INTERSECTION):
            for j, v in enumerate(Sp):
                if support == SUPPORT_INTERSECTION and v not in Sq:
                    continue
                lp.append(s_logp[m][j])
                lq.append(t_at_s[m][j])
        if support in (SUPPORT_UNION, SUPPORT_TEACHER):
            for j, v in enumerate(Sq):
                if support == SUPPORT_UNION and v in Sp:
                    continue
                lp.append(s_at_t[m][j])
                lq.append(t_logp[m][j])
        if support not in (SUPPORT_UNION, SUPPORT_STUDENT, SUPPORT_TEACHER, SUPPORT_INTERSECTION):
            raise ValueError("unknown support")
        rev, fwd = _kl_pair(lp, lq)
        out["kl_rev"][m], out["kl_fwd"][m] = rev, fwd
        out["loss"][m] = _row_loss(rev, fwd, int(src[m]), loss_mode)
        out["overlap"][m] = len(set(Sp) & set(Sq)) / K
    if cu is not None:
        out["seq_loss"], out["t_ratio"] = _segments(out["loss"], src, cu)
    return out


# ---------------------------------------------------------------------------
# The proposer's decode steps (Section 3.2.3, propose stage)
# ---------------------------------------------------------------------------

def propose_decode(steps, k_cache, v_cache, page_table, ctx_lens, scale, W, K, seq_ids=None):
    """The driver's draft of gamma tokens, one autoregressive step at a time
    (Section 3.2.3: the driver proposes gamma tokens; Eq. (9): the draft is
    drawn from the driver's own distribution at temperature 1, Appendix A).

    Step j of sequence b (b over ``seq_ids``, default all) appends its input
    token's keys/values at position L_b + j of the proposer's own paged cache,
    attends over keys 0 .. L_b + j (a one-row window), scores the row with the
    LM head and draws the next token by inverse CDF with the uniform u[b].
    ``steps`` is a list of dicts with q [n,Hq,D], k_new / v_new [n,Hkv,D],
    hidden [n,Hd] and u [n] (n = number of sequences handled, row i for the
    i-th of the ascending ``seq_ids``): the inputs a
    full model derives from the previous step's token through layers that
    are not part of this path.

    Returns (per-step list of dicts out / lm / token, k_cache', v_cache').
    """
    kc = np.array(k_cache, copy=True)
    vc = np.array(v_cache, copy=True)
    seqs = list(range(len(ctx_lens))) if seq_ids is None else [int(b) for b in seq_ids]
    if seqs != sorted(set(seqs)):
        raise ValueError("seq_ids must be ascending and distinct (row i is seq_ids[i])")
    n = len(seqs)
    sid = np.asarray(seqs, np.int64)
    res = []
    for j, st in enumerate(steps):
        lens = np.asarray(ctx_lens, np.int64).copy()
        lens[sid] += j
        # cu_q indexes the handled sequences' rows: row i belongs to seqs[i]
        cu_full = np.zeros(len(ctx_lens) + 1, np.int64)
        for i, b in enumerate(seqs):
            cu_full[b + 1] = 1
        cu_full = np.cumsum(cu_full)
        out, kc, vc = verify_attn_paged(st["q"], st["k_new"], st["v_new"], kc, vc, page_table,
                                        lens, cu_full, scale, seq_ids=sid, n_seq=n)
        logits = logits_fp64(st["hidden"], W)
        lm = lmhead_logsoftmax(st["hidden"], W, np.zeros(n, np.int64), K, logits=logits)
        draws = [sample_categorical(logits[i], float(st["u"][i])) for i in range(n)]
        res.append({"out": out, "lm": lm, "token": np.array([d[0] for d in draws]),
                    "margin": np.array([d[1] for d in draws]), "logits": logits})
    return res, kc, vc
