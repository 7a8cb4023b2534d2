"""Argus's prompt-routing control plane on the CPU: the Optimized Distribution
Aligner (ODA) that turns the demand histogram H and the solver's load split F into
the Probabilistic Approximation Shift Map (PASM), the quality-degradation objective
it minimises, the scheduler's draw from the PASM, and the greedy worker selector.

Test infrastructure only (see the package docstring).

Levels are indexed 0 .. n-1 from the slowest / most accurate (v_1 in the paper) to
the fastest / most approximate (v_n).
"""

import numpy as np


def oda(H, F):
    """ODA, Alg. 1 (Sec. 4.3). H[i]: share of prompts whose optimal level is i (the
    classifier's preference histogram); F[i]: share of the load the solver assigns to
    level i (sum H = sum F). Returns the PASM T with T[i][j] = probability that a
    prompt whose optimal level is i is served at level j.

    The levels are visited from the fastest to the slowest. At level i:
    * H(i) > F(i): the excess H(i) - F(i) moves one level to the left (slower, so no
      quality loss); the step probability (H(i) - F(i)) / H(i) applies to all mass
      currently at i, including mass that arrived from the right;
    * otherwise, while H(i) < F(i): take min(H(i - m), F(i) - H(i)) from the levels on
      the left, nearest first (m = 1, 2, ...), each shift divided by H_old(i - m).
    The final PASM is the composition of the step probabilities along each path
    (the product formula after Alg. 1); the composition is carried out here by keeping,
    at every level, how much of its current mass originated at each level: a step
    probability moves the same fraction of every origin's share."""
    H_old = np.asarray(H, dtype=np.float64).copy()
    Fv = np.asarray(F, dtype=np.float64)
    n = H_old.size
    if Fv.size != n or n == 0:
        raise ValueError("H and F must have the same, non-zero length")
    if (H_old < 0).any() or (Fv < 0).any():
        raise ValueError("histograms must be non-negative")
    if abs(H_old.sum() - Fv.sum()) > 1e-9 * max(1.0, H_old.sum()):
        raise ValueError("H and F must have the same total")
    # mass[k][o]: mass now at level k that originated at level o
    mass = np.diag(H_old)
    Hc = H_old.copy()
    for i in range(n - 1, -1, -1):
        if Hc[i] > Fv[i]:
            if i == 0:
                # the slowest level: the totals agree, so only rounding can be left over
                continue
            frac = (Hc[i] - Fv[i]) / Hc[i]
            moved = frac * mass[i]
            mass[i - 1] += moved
            mass[i] -= moved
            Hc[i - 1] += Hc[i] - Fv[i]
            Hc[i] = Fv[i]
        else:
            m = 1
            while Hc[i] < Fv[i] and i - m >= 0:
                shift = min(Hc[i - m], Fv[i] - Hc[i])
                if shift > 0:
                    # levels on the left hold only their own prompts at this point
                    mass[i][i - m] += shift
                    mass[i - m][i - m] -= shift
                    Hc[i - m] -= shift
                    Hc[i] += shift
                m += 1
    T = np.zeros((n, n))
    for o in range(n):
        if H_old[o] > 0:
            T[o] = mass[:, o] / H_old[o]
        else:
            T[o, o] = 1.0
    return T


def degradation(T, H, D):
    """Eq. 2: sum over i and over faster levels j > i of P(j | i) H(i) D(j, i), with
    D[j][i] the profiled quality loss of serving a level-i prompt at level j."""
    T = np.asarray(T, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    n = H.size
    return float(sum(T[i, j] * H[i] * D[j, i] for i in range(n) for j in range(i + 1, n)))


def route(T, level, u):
    """Prompt Scheduler (Sec. 4.4): the level a prompt whose optimal level is `level`
    is sent to, drawn from the PASM row with the uniform number u in [0, 1): the first
    j (from the slowest) whose cumulative probability exceeds u; the last level with
    positive probability when rounding leaves the row's sum at or below u."""
    row = np.asarray(T, dtype=np.float64)[level]
    c = 0.0
    last = level
    for j in range(row.size):
        if row[j] > 0:
            last = j
        c += row[j]
        if u < c:
            return j
    return last


def select_worker(queue_len, t_proc, worker_level, level):
    """Worker selector, Eq. 3 (Sec. 4.4): among the workers running `level`, the one
    minimising (queued requests) x (generation time at that level), lowest worker
    index on ties; -1 when no worker runs the level."""
    best, best_cost = -1, None
    for w in range(len(worker_level)):
        if worker_level[w] != level:
            continue
        cost = float(queue_len[w]) * float(t_proc[w])
        if best_cost is None or cost < best_cost:
            best, best_cost = w, cost
    return best
