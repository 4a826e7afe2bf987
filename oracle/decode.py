"""Oracle of the per-step decision rules and the gated block decode (test infrastructure only).

Notation follows Section 3 ("Diffusion Decoding Setup", "Confidence-Oriented
Residual Acceptance"): canvas x, unresolved set U, prediction x_hat, confidence
c, persistence counter m, transfer set T, accepted set A.

State arrays (per batch row b, canvas position i):
    tokens[b, i]      canvas x (mask id where masked)
    unresolved[b, i]  1 iff i in U
    prev_top1[b, i]   x_hat of the previous executed step, -1 = none
    persist[b, i]     counter m
    block_idx[b]      active generation block (== n_blocks once finished)
    step_idx[b]       executed steps so far in the active block

Readings of points the paper leaves open, numbered as in the rest of the oracle:
    R1  k_s: linear split of the block's M masked positions over S_b steps,
        k_s = floor(M / S_b) + [s < M mod S_b], fixed at block start.
    R2  the transfer rule takes the k_s highest-confidence positions of the
        active block; equal confidence -> lower position first.
    R3  candidates are U restricted to the active block.
    R4  order in a step: scores -> counter update -> T -> A on (U \\ T) -> commit -> terminate.
    R5  persistence scope.  BLOCK (default): counters and previous top-1 reset when a
        block becomes active (its first executed step), so only the active block is
        scored.  GLOBAL: every unresolved generation position is scored on every
        executed pass and its counter runs across blocks without a reset; transfer and
        gate still act on the active block only, so a block whose positions already
        persisted during earlier blocks can end after one pass.
    R7  both gate comparisons inclusive; the confidence test and the transfer
        ranking are taken on c rounded to fp32, against fp32(delta_p).
    R9  argmax ties -> lowest token id.  R10  the mask id is never predicted.
    R13 gate disabled -> A is empty (the original decoder).
    R27 EOS-aware controller (EoTP, Table 2): after a step's commits, the lowest
        committed EOS of the generation region cuts the canvas.  Unresolved positions
        after it are resolved as EOS (the suffix is removed; committed tokens keep their
        value).  The active block still decodes its positions before the EOS, then the row
        stops: no later block is executed.
"""
import numpy as np

NONE = -1


# --- Eq. (1) -----------------------------------------------------------------------------
def top1_confidence(logits, mask_id=None):
    """x_hat = argmax_v p_v and c = max_v p_v with p = softmax(logits), per row (Eq. 1).

    logits [..., V].  The mask-id column is excluded (R10).  Ties go to the lowest
    token id (R9): np.argmax returns the first maximum.  fp64 throughout."""
    l = np.array(logits, dtype=np.float64, copy=True)
    if mask_id is not None:
        l[..., mask_id] = -np.inf
    p = np.exp(l - np.max(l, axis=-1, keepdims=True))
    p = p / np.sum(p, axis=-1, keepdims=True)
    x_hat = np.argmax(p, axis=-1)
    c = np.take_along_axis(p, x_hat[..., None], axis=-1)[..., 0]
    return x_hat.astype(np.int64), c


# --- Eq. (2) -----------------------------------------------------------------------------
def persistence_update(prev, m, x_hat):
    """m^(s) = m^(s-1) + 1 if x_hat^(s) == x_hat^(s-1) else 0 (Eq. 2).

    At a position's first executed step there is no previous prediction
    (prev == NONE) and the counter is zero.  Returns (new_prev, new_m)."""
    same = (prev != NONE) & (prev == x_hat)
    return np.asarray(x_hat).copy(), np.where(same, m + 1, 0)


# --- transfer schedule and rule (R1, R2) -------------------------------------------------
def transfer_schedule(M, S):
    """k_s for s = 0..S-1: the block's M masked positions split as evenly as possible,
    the remainder going to the earliest steps (R1).  sum(k) == M."""
    base, rem = divmod(int(M), int(S))
    return np.array([base + (1 if s < rem else 0) for s in range(S)], dtype=np.int64)


def transfer_set(candidates, c32, k):
    """Original low-confidence rule: the min(k, |candidates|) candidates of highest
    confidence; ties -> lower position (R2).  candidates: position array; c32: fp32
    confidences indexed by position.  Returns a sorted position array."""
    candidates = np.asarray(candidates)
    if len(candidates) == 0 or k <= 0:
        return np.zeros(0, dtype=np.int64)
    order = sorted(candidates.tolist(), key=lambda i: (-float(c32[i]), i))
    return np.array(sorted(order[:min(int(k), len(order))]), dtype=np.int64)


# --- Eq. (3) -----------------------------------------------------------------------------
def gate_accept(c32, m, delta_p, m_req):
    """a_i = 1[c_i >= delta_p and m_i >= m] (Eq. 3), both comparisons inclusive (R7)."""
    return (np.asarray(c32, dtype=np.float32) >= np.float32(delta_p)) & (np.asarray(m) >= m_req)


# --- one denoising step on one batch row ---------------------------------------------------
def step_row(st, b, logits_blk, prompt_len, block_len, steps_per_block, n_blocks, mask_id,
             delta_p, m_req, gate_enabled, k_override=None, logits_row0=None, scope="block",
             eos_id=None):
    """Apply the decision part of one executed step to batch row b, in place.

    logits_blk [n_rows, V] are the logits of canvas rows starting at `logits_row0`
    (default: the active block's first position).  scope "block" or "global" (R5); the
    global scope needs rows covering every unresolved position.  Returns a dict with
    x_hat, c, c32 for those rows, and T, A, done for the block."""
    blk = int(st["block_idx"][b])
    if blk >= n_blocks:                       # row already finished all blocks
        return {"finished": True, "T": np.zeros(0, np.int64), "A": np.zeros(0, np.int64),
                "done": True}
    lo = prompt_len + blk * block_len
    pos = np.arange(lo, lo + block_len)
    s = int(st["step_idx"][b])
    if scope == "block" and s == 0:           # R5: the block becomes active
        st["prev_top1"][b, pos] = NONE
        st["persist"][b, pos] = 0

    row0 = lo if logits_row0 is None else logits_row0
    x_hat_rows, c_rows = top1_confidence(logits_blk, mask_id)              # Eq. (1)
    scored = np.arange(row0, row0 + len(x_hat_rows))
    x_hat = np.full(st["tokens"].shape[1], NONE, dtype=np.int64)
    c = np.zeros(st["tokens"].shape[1], dtype=np.float64)
    x_hat[scored] = x_hat_rows
    c[scored] = c_rows
    c32 = c.astype(np.float32)

    U_blk = pos[st["unresolved"][b, pos] == 1]                             # R3
    if scope == "global":                     # R5: every scored unresolved position
        U_upd = scored[st["unresolved"][b, scored] == 1]
        unscored = np.setdiff1d(np.nonzero(st["unresolved"][b])[0], scored)
        assert len(unscored) == 0, "global scope needs scores for every unresolved position"
    else:
        U_upd = U_blk
    new_prev, new_m = persistence_update(st["prev_top1"][b, U_upd],       # Eq. (2)
                                         st["persist"][b, U_upd], x_hat[U_upd])
    st["prev_top1"][b, U_upd] = new_prev
    st["persist"][b, U_upd] = new_m

    M = block_len                              # R1: the block starts fully masked
    k = transfer_schedule(M, steps_per_block)[s] if k_override is None else k_override
    T = transfer_set(U_blk, c32, k)                                        # R2
    residual = np.setdiff1d(U_blk, T)
    if gate_enabled:                                                       # Eq. (3), R13
        ok = gate_accept(c32[residual], st["persist"][b, residual], delta_p, m_req)
        A = residual[ok]
    else:
        A = np.zeros(0, dtype=np.int64)

    fixed = np.union1d(T, A)                                               # Eq. (4)
    st["tokens"][b, fixed] = x_hat[fixed]
    st["unresolved"][b, fixed] = 0
    removed, cut = np.zeros(0, dtype=np.int64), None
    if eos_id is not None:                                                 # R27
        L = st["tokens"].shape[1]
        gen = np.arange(prompt_len, L)
        eos = gen[(st["unresolved"][b, gen] == 0) & (st["tokens"][b, gen] == eos_id)]
        if len(eos):
            cut = int(eos.min())
            later = np.arange(cut + 1, L)
            removed = later[st["unresolved"][b, later] == 1]
            st["tokens"][b, removed] = eos_id
            st["unresolved"][b, removed] = 0
    done = not st["unresolved"][b, pos].any()                              # termination
    st["step_idx"][b] = s + 1
    if done:
        st["block_idx"][b] = n_blocks if cut is not None else blk + 1
        st["step_idx"][b] = 0
    return {"finished": False, "x_hat": x_hat_rows, "c": c_rows, "c32": c_rows.astype(np.float32),
            "T": T, "A": A, "done": done, "block": blk, "step": s, "k": int(k),
            "residual": residual, "m": st["persist"][b].copy(),
            "removed": removed, "eos_cut": cut}


def block_positions(st, b, prompt_len, block_len, n_blocks):
    blk = min(int(st["block_idx"][b]), n_blocks - 1)
    lo = prompt_len + blk * block_len
    return np.arange(lo, lo + block_len)


def copy_state(st):
    return {k: np.array(v, copy=True) for k, v in st.items()}


# --- the gated block decode (Fig. 2; Section 3, "From acceptance to runtime") -----------
def block_decode(logits_fn, prompt, gen_len, mask_id, block_len, steps_per_block,
                 delta_p, m_req, gate_enabled, record=False, scope="block", eos_id=None):
    """Decode every batch row independently (R15), block by block, left to right.

    logits_fn(tokens [B, L], rows list-of-arrays) -> list of [len(rows_b), V] logits.
    Each executed step runs one dense pass, then the decision rules; a block ends
    once it holds no unresolved position, skipping its remaining passes.  The block
    scope scores the active block's rows, the global scope the whole generation
    region (R5).  eos_id enables the EOS-aware controller (R27).

    Returns (tokens [B, L], passes [B, n_blocks], trace) where trace holds the
    pre-step state and step outputs of every executed pass when record=True."""
    prompt = np.asarray(prompt)
    B, P = prompt.shape
    L = P + gen_len
    n_blocks = gen_len // block_len
    st = {
        "tokens": np.full((B, L), mask_id, dtype=np.int64),
        "unresolved": np.zeros((B, L), dtype=np.uint8),
        "prev_top1": np.full((B, L), NONE, dtype=np.int64),
        "persist": np.zeros((B, L), dtype=np.int64),
        "block_idx": np.zeros(B, dtype=np.int64),
        "step_idx": np.zeros(B, dtype=np.int64),
    }
    st["tokens"][:, :P] = prompt
    st["unresolved"][:, P:] = 1
    passes = np.zeros((B, n_blocks), dtype=np.int64)
    trace = []
    while (st["block_idx"] < n_blocks).any():
        active = [b for b in range(B) if st["block_idx"][b] < n_blocks]
        if scope == "global":
            rows = [np.arange(P, L) for _ in range(B)]
        else:
            rows = [block_positions(st, b, P, block_len, n_blocks) for b in range(B)]
        pre = copy_state(st) if record else None
        logits = logits_fn(st["tokens"].copy(), rows)
        outs = {}
        for b in active:
            blk = int(st["block_idx"][b])
            outs[b] = step_row(st, b, logits[b], P, block_len, steps_per_block, n_blocks,
                               mask_id, delta_p, m_req, gate_enabled,
                               logits_row0=int(rows[b][0]), scope=scope, eos_id=eos_id)
            passes[b, blk] += 1
        if record:
            trace.append({"pre": pre, "rows": rows, "logits": logits, "out": outs})
    return st["tokens"], passes, trace


def dense_endpoint(logits_fn, prompt, gen_len, mask_id, block_len, steps_per_block,
                   eos_id=None):
    """Y*: the original fixed-horizon decoder = the block decode with the gate disabled
    (with eos_id: the EOS-aware dense decoder, R27)."""
    tokens, passes, _ = block_decode(logits_fn, prompt, gen_len, mask_id, block_len,
                                     steps_per_block, 1.0, 0, gate_enabled=False, eos_id=eos_id)
    return tokens, passes
