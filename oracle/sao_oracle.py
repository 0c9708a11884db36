"""fp64 CPU oracle of the SAO per-token training-loss pass.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Every quantity of the pass is a closed-form function of its inputs, so each
function below is the plain definition evaluated in float64, in the order the
paper states it:

* ``token_logprob``  -- log pi_theta(a_t|s_t) of the LM head at temperature 1
  over the full vocabulary (Sec. 3.1, Eq. 1-2; evaluation settings of Sec. 4.1).
* ``advantage``      -- skip-observation token-level GAE (Sec. 3.2, Eq. 4-5)
  with the length-adaptive lambda_policy = 1 - 1/(alpha*l) and critic returns
  at lambda_critic = 1 (Sec. 4.1, training details); textbook GAE of Sec. 2 is
  the special case without observations.
* ``dis_loss``       -- the direct double-sided importance-sampling objective:
  ratio against the rollout log-probs (Eq. 2), calibration f with strict band
  edges (Eq. 3), token-level mean of f(r) A log pi (Eq. 1).
* ``loss_backward``  -- gradient of that objective into the hidden states and
  the head weights through the log-softmax.
* ``value_forward`` / ``value_loss`` -- a bias-free H->1 critic head and the
  critic's squared-error loss against the returns (Sec. 2, PPO paragraph).
* ``ppo_loss``       -- the comparison objectives the paper sets DIS against:
  the clipped surrogate of Sec. 2 (symmetric, or clip-higher with
  eps_high != eps_low) and the decoupled three-policy form of Sec. 3.1, where
  pi_old / pi_rollout weighs the clipped term.
* ``explained_variance`` -- EV = 1 - Var(R - V) / Var(R), the critic diagnostic
  of Sec. 4.4, over the loss-mask tokens.
* ``step_advantage``   -- the step-level GAE of App. A.1: one advantage per
  agentic step, with the step value as the mean or the last of its token values
  and lambda scaled by the number of steps.
* ``group_advantage`` / ``running_mean_advantage`` -- the critic-free baselines
  the paper compares with: GRPO's group-normalised sequence reward (Sec. 2)
  and a sliding-window running-mean reward baseline (the 8 most recent rewards
  of each prompt in the Sec. 4.3 ablation, the 128 most recent in the Sec. 4.5
  online comparison), one advantage per trajectory.

Readings where the paper is silent (all listed in the design notes):
  gamma defaults to 1; ``l`` in lambda_policy is the trajectory's token length
  (observations included), lambda clamped at 0; rewards on observation tokens
  fold into the preceding action, rewards before the first action are dropped;
  the value after a trajectory's last action is 0; the token mean divides by
  N = number of loss-mask tokens (clipped ones included); f(r) is a
  stop-gradient weight; the library minimises -L; band edges are strict as in
  Eq. 3 (equality is clipped); a NaN ratio is flagged non-finite and
  contributes exactly 0. For the comparison objectives: the same token mean
  and N as DIS; a token is clipped exactly when A > 0 and r > 1 + eps_high or
  A < 0 and r < 1 - eps_low (strict, as Sec. 3.1 states standard clipping);
  the pi_old / pi_rollout weight is a stop-gradient constant and is not
  truncated; EV uses population variances over loss-mask tokens and is NaN
  when there are none or Var(R) = 0. A step of App. A.1 is a maximal run of
  consecutive loss-mask tokens inside one trajectory (one model turn); the
  step reward sums the rewards from the step's first token up to the next
  step's first token (or the trajectory's end), so observation rewards fold
  into the preceding step as in the token-level form. For the critic-free
  baselines: a trajectory's reward is the sum of its token rewards; a group is
  `group_size` consecutive trajectories; sigma uses the population variance
  with eps_stab inside the root, as printed; the running-mean window holds the
  `window` most recent earlier rewards of the same key (prompt), the
  trajectory's own reward excluded, in arrival order (history first, then the
  batch in order), and an empty window gives baseline 0.

Large inputs are processed in blocks of rows only to bound memory: rows are
independent in every definition here, so the blocking changes no arithmetic.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np

FLAG_MASKED, FLAG_USED, FLAG_LOW, FLAG_HIGH, FLAG_NONFINITE = 0, 1, 2, 3, 4


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _active_rows(T: int, mask, rows):
    if rows is not None:
        return np.asarray(rows, dtype=np.int64)
    if mask is None:
        return np.arange(T, dtype=np.int64)
    return np.nonzero(np.asarray(mask) != 0)[0].astype(np.int64)


# --------------------------------------------------------------------------- #
# Eq. (1)-(2): per-token log-probability under the current policy's LM head.
# --------------------------------------------------------------------------- #
def token_logprob(hidden, w_head, target, mask=None, rows: Optional[Sequence[int]] = None,
                  block: int = 1024, w64: Optional[np.ndarray] = None):
    """log pi(y_t | s_t) = z_{t,y_t} - log sum_v exp(z_{t,v}),  z_{t,v} = h_t . W_v.

    Returns ``(logp, lse)`` as float64 arrays of length T. Rows outside the loss
    mask (or outside ``rows`` when given) are 0, matching the library's
    convention for rows it does not compute.
    """
    T = hidden.shape[0]
    W = _f64(w_head) if w64 is None else w64
    tgt = np.asarray(target, dtype=np.int64)
    logp = np.zeros(T, dtype=np.float64)
    lse = np.zeros(T, dtype=np.float64)
    act = _active_rows(T, mask, rows)
    for s in range(0, act.size, block):
        r = act[s:s + block]
        z = _f64(hidden[r]) @ W.T                              # z_{t,v} = sum_k h_{t,k} W_{v,k}
        if np.abs(z).max(initial=0.0) > 700.0:
            raise ValueError("logits beyond the range where exp() is finite in float64")
        lse_r = np.log(np.exp(z).sum(axis=1))                  # log sum_v exp(z_{t,v})
        lse[r] = lse_r
        logp[r] = z[np.arange(r.size), tgt[r]] - lse_r         # z_{t,y_t} - lse_t
    return logp, lse


def token_logprob_loop(hidden, w_head, target, mask=None):
    """The same definition as ``token_logprob`` written as scalar loops (tiny inputs)."""
    T, H = hidden.shape
    V = w_head.shape[0]
    logp = [0.0] * T
    lse = [0.0] * T
    for t in range(T):
        if mask is not None and not mask[t]:
            continue
        h = [float(x) for x in hidden[t]]
        zs = []
        for v in range(V):
            w = w_head[v]
            zs.append(math.fsum(h[k] * float(w[k]) for k in range(H)))
        s = math.fsum(math.exp(z) for z in zs)
        lse[t] = math.log(s)
        logp[t] = zs[int(target[t])] - lse[t]
    return np.array(logp), np.array(lse)


# --------------------------------------------------------------------------- #
# Eq. (4)-(5): skip-observation token-level GAE, with critic returns.
# --------------------------------------------------------------------------- #
def trajectory_lambda(L_tokens: int, n_actions: int, lam: float, alpha: float,
                      length: str = "tokens") -> float:
    """lambda_policy = 1 - 1/(alpha*l) (length-adaptive GAE, Sec. 4.1), clamped at 0.

    ``alpha <= 0`` selects the fixed ``lam``. ``l`` is the trajectory's token
    length by default; ``length="actions"`` uses the number of action tokens.
    """
    if alpha <= 0.0:
        return float(lam)
    l = L_tokens if length == "tokens" else n_actions
    if l <= 0:
        return 0.0
    return max(0.0, 1.0 - 1.0 / (alpha * l))


def advantage(values, rewards, mask, cu_seqlens, gamma: float = 1.0, lam: float = 1.0,
              alpha: float = 0.0, length: str = "tokens"):
    """Skip-observation GAE advantages and lambda=1 returns for a packed batch.

    For trajectory b with action positions tau_0 < ... < tau_{n-1} (mask 1) in
    [s_b, e_b), and tau_n := e_b:
        r~_k   = sum of rewards at positions tau_k .. tau_{k+1}-1
        delta_k = r~_k + gamma * V(tau_{k+1}) - V(tau_k)     (V after the last action = 0)
        A_k     = delta_k + gamma * lambda_b * A_{k+1}        (A_n = 0)          Eq. (4)-(5)
        G_k     = r~_k + gamma * G_{k+1}                      (G_n = 0, lambda_critic = 1)
    Outputs are float64 arrays with 0 at mask-0 positions, and N = sum(mask).
    """
    vals, rew = _f64(values), _f64(rewards)
    m = np.asarray(mask) != 0
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    T = vals.shape[0]
    adv = np.zeros(T, dtype=np.float64)
    ret = np.zeros(T, dtype=np.float64)
    for b in range(cu.size - 1):
        s, e = int(cu[b]), int(cu[b + 1])
        tau = [t for t in range(s, e) if m[t]]
        n = len(tau)
        if n == 0:
            continue
        lam_b = trajectory_lambda(e - s, n, lam, alpha, length)
        bounds = tau + [e]
        r_fold = [math.fsum(rew[bounds[k]:bounds[k + 1]]) for k in range(n)]
        v = [vals[t] for t in tau] + [0.0]
        A_next, G_next = 0.0, 0.0
        for k in range(n - 1, -1, -1):
            delta = r_fold[k] + gamma * v[k + 1] - v[k]
            A_k = delta + gamma * lam_b * A_next
            G_k = r_fold[k] + gamma * G_next
            adv[tau[k]], ret[tau[k]] = A_k, G_k
            A_next, G_next = A_k, G_k
    return adv, ret, int(m.sum())


# --------------------------------------------------------------------------- #
# Eq. (1)-(3): direct double-sided importance sampling and the token mean.
# --------------------------------------------------------------------------- #
def dis_loss(logp, logp_rollout, adv, mask, eps_low, eps_high, n_tokens: Optional[int] = None):
    """DIS loss, its gradient w.r.t. log pi, per-token flags and counts.

    eps_low/eps_high are the float32 values the library receives, widened to
    float64. For each loss-mask token:
        rho_t = exp(log pi_t - log pi_rollout_t)                         Eq. (2)
        flag  = 4 if rho is NaN; 2 if rho <= lo; 3 if rho >= 1+eps_high; else 1
        c_t   = [flag == 1]                    (strict band of f, Eq. (3))
    with lo = max(0, 1 - eps_low): a ratio is never negative, so eps_low >= 1 leaves
    only rho = 0 (pi = 0, or exp underflow) below the band, and that token is
    clipped low like any ratio at the edge rather than weighting log pi = -inf by 0.
    With N the token-mean denominator:
        loss[0] = -(1/N) sum_t c_t rho_t A_t log pi_t    (minus Eq. (1))
        loss[1] = -(1/N) sum_t c_t rho_t A_t             (same gradient, f as stop-gradient)
        g_t     = -c_t rho_t A_t / N                     (d loss / d log pi_t; exactly 0 if c_t=0)
    counts = [sum(mask), used, clipped-low, clipped-high, non-finite].
    """
    lp, lro, A = _f64(logp), _f64(logp_rollout), _f64(adv)
    m = np.asarray(mask) != 0
    lo_edge = max(0.0, 1.0 - float(np.float32(eps_low)))
    hi_edge = 1.0 + float(np.float32(eps_high))
    N = int(m.sum()) if n_tokens is None else int(n_tokens)
    with np.errstate(over="ignore", invalid="ignore"):
        rho = np.exp(lp - lro)                                   # Eq. (2)
    flags = np.where(np.isnan(rho), FLAG_NONFINITE,
             np.where(rho <= lo_edge, FLAG_LOW,
              np.where(rho >= hi_edge, FLAG_HIGH, FLAG_USED)))
    flags = np.where(m, flags, FLAG_MASKED).astype(np.uint8)
    used = flags == FLAG_USED                                    # 1 - eps_l < rho < 1 + eps_h
    g = np.zeros(lp.shape[0], dtype=np.float64)
    loss = np.zeros(2, dtype=np.float64)
    if N > 0:
        idx = np.nonzero(used)[0]
        loss[0] = -math.fsum(rho[idx] * A[idx] * lp[idx]) / N
        loss[1] = -math.fsum(rho[idx] * A[idx]) / N
        g[idx] = -rho[idx] * A[idx] / N
    counts = np.array([int(m.sum()), int(used.sum()), int((flags == FLAG_LOW).sum()),
                       int((flags == FLAG_HIGH).sum()), int((flags == FLAG_NONFINITE).sum())],
                      dtype=np.int64)
    return loss, g, flags, counts


# --------------------------------------------------------------------------- #
# Backward through the log-softmax into hidden states and head weights.
# --------------------------------------------------------------------------- #
def loss_backward(hidden, w_head, target, lse, g, dh_rows: Optional[Sequence[int]] = None,
                  dw_rows: Optional[Sequence[int]] = None, block: int = 1024,
                  w64: Optional[np.ndarray] = None):
    """dz_{t,v} = g_t (1[v = y_t] - exp(z_{t,v} - lse_t));  dH_t = sum_v dz_{t,v} W_v;
    dW_v = sum_t dz_{t,v} h_t.

    Only rows with g_t != 0 contribute; dH is exactly 0 elsewhere. ``dh_rows``
    restricts dH to the given token rows (others 0) and ``dw_rows`` restricts dW
    to the given vocabulary rows (others 0); both default to everything.
    Returns float64 ``(dH [T,H], dW [V,H])``.
    """
    T, H = hidden.shape
    W = _f64(w_head) if w64 is None else w64
    V = W.shape[0]
    gg, L = _f64(g), _f64(lse)
    tgt = np.asarray(target, dtype=np.int64)
    live = np.nonzero(gg != 0.0)[0]
    dH = np.zeros((T, H), dtype=np.float64)
    dW = np.zeros((V, H), dtype=np.float64)

    want_dh = live if dh_rows is None else np.intersect1d(live, np.asarray(dh_rows, dtype=np.int64))
    for s in range(0, want_dh.size, block):
        r = want_dh[s:s + block]
        z = _f64(hidden[r]) @ W.T
        dz = -gg[r, None] * np.exp(z - L[r, None])
        dz[np.arange(r.size), tgt[r]] += gg[r]
        dH[r] = dz @ W

    vrows = np.arange(V, dtype=np.int64) if dw_rows is None else np.asarray(dw_rows, dtype=np.int64)
    Wv = W[vrows]
    for s in range(0, live.size, block):
        r = live[s:s + block]
        h = _f64(hidden[r])
        z = h @ Wv.T                                           # z_{t,v} for the requested v
        dz = -gg[r, None] * np.exp(z - L[r, None])
        onehot = tgt[r, None] == vrows[None, :]
        dz += onehot * gg[r, None]
        dW[vrows] += dz.T @ h
    return dH, dW


def loss_backward_loop(hidden, w_head, target, lse, g):
    """``loss_backward`` as scalar loops (tiny inputs)."""
    T, H = hidden.shape
    V = w_head.shape[0]
    dH = np.zeros((T, H))
    dW = np.zeros((V, H))
    for t in range(T):
        if g[t] == 0.0:
            continue
        h = [float(x) for x in hidden[t]]
        for v in range(V):
            w = [float(x) for x in w_head[v]]
            z = math.fsum(h[k] * w[k] for k in range(H))
            dz = float(g[t]) * ((1.0 if v == int(target[t]) else 0.0) - math.exp(z - float(lse[t])))
            for k in range(H):
                dH[t, k] += dz * w[k]
                dW[v, k] += dz * h[k]
    return dH, dW


def surrogate_S(hidden, w_head, target, logp_rollout, adv, used, n_tokens: int):
    """S = -(1/N) sum_{used t} exp(log pi_t - log pi_rollout_t) A_t with the used set frozen.

    Its gradient equals the gradient of -Eq. (1) with f(r) as a stop-gradient
    weight; finite differences of S pin ``loss_backward``.
    """
    rows = np.nonzero(np.asarray(used))[0]
    lp, _ = token_logprob(hidden, w_head, target, rows=rows)
    rho = np.exp(lp[rows] - _f64(logp_rollout)[rows])
    return -math.fsum(rho * _f64(adv)[rows]) / n_tokens


# --------------------------------------------------------------------------- #
# Critic head and its squared-error loss (Sec. 2, PPO paragraph).
# --------------------------------------------------------------------------- #
def value_forward(hidden, w_value):
    """v_t = h_t . w_v (bias-free H->1 head)."""
    return _f64(hidden) @ _f64(w_value)


def value_loss(hidden, w_value, v, ret, mask, n_tokens: Optional[int] = None):
    """L_V = (1/N) sum_t m_t (v_t - G_t)^2, with its gradients.

    Returns ``(L_V, dH_v [T,H], dw_v [H])`` where dv_t = 2 m_t (v_t - G_t) / N,
    dH_v = dv_t w_v and dw_v = sum_t dv_t h_t.
    """
    vv, G = _f64(v), _f64(ret)
    m = (np.asarray(mask) != 0).astype(np.float64)
    N = int(m.sum()) if n_tokens is None else int(n_tokens)
    if N == 0:
        return 0.0, np.zeros(hidden.shape), np.zeros(hidden.shape[1])
    diff = vv - G
    L = math.fsum(m * diff * diff) / N
    dv = 2.0 * m * diff / N
    dH = dv[:, None] * _f64(w_value)[None, :]
    dw = _f64(hidden).T @ dv
    return L, dH, dw


# --------------------------------------------------------------------------- #
# Comparison objectives: the clipped surrogate of Sec. 2 and decoupled PPO.
# --------------------------------------------------------------------------- #
def ppo_loss(logp, logp_old, adv, mask, eps_low, eps_high, n_tokens: Optional[int] = None,
             logp_behav=None):
    """Clipped-surrogate loss, its gradient w.r.t. log pi, per-token flags and counts.

    The unified objective of Sec. 2 with separate lower and upper clip widths
    (eps_low == eps_high is standard PPO, eps_high > eps_low is clip-higher),
    as a token mean with the same N as the DIS loss. For each loss-mask token:
        r_t   = exp(log pi_t - log pi_old_t)          (the Sec. 2 ratio)
        w_t   = exp(log pi_old_t - log pi_behav_t)     (decoupled form of Sec. 3.1; 1 without behav)
        flag  = 4 if r or w is NaN;
                3 if A_t > 0 and r_t > 1 + eps_high;  2 if A_t < 0 and r_t < 1 - eps_low;  else 1
        term  = w_t * min(r_t A_t, clip(r_t, 1 - eps_low, 1 + eps_high) A_t)
    The min picks the clipped product exactly on flags 2 and 3, where the term
    is a constant in log pi. Then
        loss  = -(1/N) sum_t term_t      (minus the objective; flag-4 tokens add 0)
        g_t   = -[flag 1] w_t r_t A_t / N
    counts = [sum(mask), unclipped, clipped-low, clipped-high, non-finite].
    """
    lp, lold, A = _f64(logp), _f64(logp_old), _f64(adv)
    m = np.asarray(mask) != 0
    lo_edge = 1.0 - float(np.float32(eps_low))
    hi_edge = 1.0 + float(np.float32(eps_high))
    N = int(m.sum()) if n_tokens is None else int(n_tokens)
    with np.errstate(over="ignore", invalid="ignore"):
        r = np.exp(lp - lold)
        w = np.ones_like(r) if logp_behav is None else np.exp(lold - _f64(logp_behav))
    bad = np.isnan(r) | np.isnan(w)
    flags = np.where(bad, FLAG_NONFINITE,
             np.where((A > 0) & (r > hi_edge), FLAG_HIGH,
              np.where((A < 0) & (r < lo_edge), FLAG_LOW, FLAG_USED)))
    flags = np.where(m, flags, FLAG_MASKED).astype(np.uint8)
    g = np.zeros(lp.shape[0], dtype=np.float64)
    loss = 0.0
    if N > 0:
        terms = []
        for t in np.nonzero(m & ~bad)[0]:
            lo_term, hi_term = r[t] * A[t], min(max(r[t], lo_edge), hi_edge) * A[t]
            terms.append(w[t] * min(lo_term, hi_term))
        loss = -math.fsum(terms) / N
        used = flags == FLAG_USED
        g[used] = -w[used] * r[used] * A[used] / N
    counts = np.array([int(m.sum()), int((flags == FLAG_USED).sum()), int((flags == FLAG_LOW).sum()),
                       int((flags == FLAG_HIGH).sum()), int((flags == FLAG_NONFINITE).sum())],
                      dtype=np.int64)
    return loss, g, flags, counts


# --------------------------------------------------------------------------- #
# Sec. 4.4: explained variance of the critic against the returns.
# --------------------------------------------------------------------------- #
def explained_variance(values, ret, mask):
    """EV = 1 - Var(R - V) / Var(R) over the loss-mask tokens (population variances).

    NaN when no token has mask 1 or when Var(R) is 0.
    """
    m = np.asarray(mask) != 0
    R, V = _f64(ret)[m], _f64(values)[m]
    if R.size == 0:
        return math.nan
    var_r = float(np.mean((R - R.mean()) ** 2))
    d = R - V
    var_d = float(np.mean((d - d.mean()) ** 2))
    return math.nan if var_r == 0.0 else 1.0 - var_d / var_r


# --------------------------------------------------------------------------- #
# App. A.1: step-level GAE (agentic step as the action).
# --------------------------------------------------------------------------- #
def steps_of(mask, s: int, e: int):
    """The steps of trajectory [s, e): maximal runs [a, z) of consecutive mask-1 tokens."""
    m = np.asarray(mask) != 0
    runs, t = [], s
    while t < e:
        if m[t]:
            a = t
            while t < e and m[t]:
                t += 1
            runs.append((a, t))
        else:
            t += 1
    return runs


def step_advantage(values, rewards, mask, cu_seqlens, gamma: float = 1.0, lam: float = 1.0,
                   alpha: float = 0.0, step_value: str = "average"):
    """Step-level GAE of App. A.1 for a packed batch.

    For trajectory b with steps [a_0, z_0), ..., [a_{n-1}, z_{n-1}) (a_n := e_b):
        V_i   = mean(values[a_i:z_i])  ("average")  or  values[z_i - 1]  ("last")
        R_i   = sum of rewards[a_i : a_{i+1}]
        lam_b = lam if alpha <= 0, else max(0, 1 - 1/(alpha * n))   (steps, not tokens)
        delta_i = R_i + gamma * V_{i+1} - V_i                        (V_n = 0)
        A_i   = delta_i + gamma * lam_b * A_{i+1}                     (A_n = 0)
        G_i   = R_i + gamma * G_{i+1}                                 (G_n = 0)
    Every token of step i gets adv = A_i and ret = G_i; mask-0 tokens get 0.
    Returns (adv, ret, last, N): last[t] = 1 on each step's final token (the
    critic's loss mask in the last-token form), N = sum(mask).
    """
    if step_value not in ("average", "last"):
        raise ValueError(step_value)
    vals, rew = _f64(values), _f64(rewards)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    T = vals.shape[0]
    adv = np.zeros(T, dtype=np.float64)
    ret = np.zeros(T, dtype=np.float64)
    last = np.zeros(T, dtype=np.uint8)
    for b in range(cu.size - 1):
        s, e = int(cu[b]), int(cu[b + 1])
        steps = steps_of(mask, s, e)
        n = len(steps)
        if n == 0:
            continue
        lam_b = float(lam) if alpha <= 0.0 else max(0.0, 1.0 - 1.0 / (alpha * n))
        if step_value == "average":
            V = [math.fsum(vals[a:z]) / (z - a) for a, z in steps]
        else:
            V = [vals[z - 1] for a, z in steps]
        starts = [a for a, _ in steps] + [e]
        R = [math.fsum(rew[starts[i]:starts[i + 1]]) for i in range(n)]
        A_next, G_next = 0.0, 0.0
        for i in range(n - 1, -1, -1):
            v_next = V[i + 1] if i + 1 < n else 0.0
            delta = R[i] + gamma * v_next - V[i]
            A_next = delta + gamma * lam_b * A_next
            G_next = R[i] + gamma * G_next
            a, z = steps[i]
            adv[a:z] = A_next
            ret[a:z] = G_next
            last[z - 1] = 1
    return adv, ret, last, int((np.asarray(mask) != 0).sum())


# --------------------------------------------------------------------------- #
# Critic-free baselines: GRPO's group normalisation and a running-mean window.
# --------------------------------------------------------------------------- #
def trajectory_rewards(rewards, cu_seqlens):
    """R_b = sum of the token rewards of trajectory b (a sequence-level reward)."""
    rew = _f64(rewards)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    return np.array([math.fsum(rew[cu[b]:cu[b + 1]]) for b in range(cu.size - 1)], dtype=np.float64)


def _broadcast(A, mask, cu_seqlens):
    m = np.asarray(mask) != 0
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    adv = np.zeros(m.size, dtype=np.float64)
    for b in range(cu.size - 1):
        s, e = int(cu[b]), int(cu[b + 1])
        adv[s:e] = np.where(m[s:e], A[b], 0.0)
    return adv


def group_advantage(rewards, mask, cu_seqlens, group_size: int, eps_stab: float):
    """GRPO advantage (Sec. 2): trajectories [g G, (g+1) G) answer one prompt;
        mu_g = (1/G) sum R_j,  sigma_g = sqrt((1/G) sum (R_j - mu_g)^2 + eps_stab),
        A_b = (R_b - mu_g) / sigma_g   on every loss-mask token of trajectory b.
    Returns (adv [T], A [B], R [B], N)."""
    R = trajectory_rewards(rewards, cu_seqlens)
    B, G = R.size, int(group_size)
    if G < 1 or B % G != 0:
        raise ValueError("B must be a multiple of group_size")
    A = np.zeros(B, dtype=np.float64)
    for g in range(B // G):
        Rg = R[g * G:(g + 1) * G]
        mu = math.fsum(Rg) / G
        var = math.fsum((Rg - mu) ** 2) / G
        with np.errstate(divide="ignore", invalid="ignore"):
            A[g * G:(g + 1) * G] = (Rg - mu) / np.float64(math.sqrt(var + eps_stab))
    return _broadcast(A, mask, cu_seqlens), A, R, int((np.asarray(mask) != 0).sum())


def running_mean_advantage(rewards, mask, cu_seqlens, window: int, history=None, keys=None):
    """Running-mean baseline: A_b = R_b - mean(the `window` most recent earlier rewards of
    b's key), the batch read in arrival order after `history` (a dict key -> list of past
    rewards, oldest first); an empty window gives baseline 0.
    Returns (adv [T], A [B], R [B], N, history after the batch)."""
    R = trajectory_rewards(rewards, cu_seqlens)
    hist = {k: [float(x) for x in v] for k, v in (history or {}).items()}
    A = np.zeros(R.size, dtype=np.float64)
    for b in range(R.size):
        k = 0 if keys is None else int(keys[b])
        past = hist.setdefault(k, [])
        win = past[-window:] if window > 0 else []
        base = math.fsum(win) / len(win) if win else 0.0
        A[b] = R[b] - base
        past.append(float(R[b]))
    return _broadcast(A, mask, cu_seqlens), A, R, int((np.asarray(mask) != 0).sum()), hist
