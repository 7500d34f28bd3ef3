"""Exact-rational reference for tiny J-DOB instances (test helper).

Evaluates the system model of Sec. II with Python ``Fraction`` arithmetic --
the binary64 inputs are converted exactly -- and enumerates every offloading
set and every CPU level vector of every user for every partition point and
GPU level, plus local computing.  Nothing is rounded, nothing is assumed
about decoupling or about which sets are worth trying; it is independent of
the C oracle and of the C brute force.
"""

from fractions import Fraction
from itertools import product


def _F(x):
    return x if isinstance(x, Fraction) else Fraction(float(x))


MODE_GREEDY, MODE_FIXED_EDGE, MODE_BINARY, MODE_CONTINUOUS = 1, 2, 4, 8


def solve_exact(prob, inst, suffix_only=False):
    """Minimum over the family of (s, j, offloading set) that
    ``prob.get("mode", 0)`` selects:

    0            every set (``suffix_only``: every gamma-ordered suffix);
    MODE_GREEDY  at each f_e only the set of Alg. 2: the list sorted by
                 gamma descending loses its head while f_e is below the
                 head's threshold of Eq. (18), written as a division here;
    MODE_FIXED_EDGE  f_e = f_e,max only;  MODE_BINARY  s = 0 only;
    MODE_CONTINUOUS  each CPU frequency is any f in [f_0, f_{K-1}]: the
                 energy kappa f^2 C grows with f, so a user's optimum is the
                 slowest f that finishes in time, C / budget, raised to f_0
                 (Eq. (20) and its clamp), solved in closed form per user.
    Local computing is always a candidate, ranked last among equal energies.
    Heterogeneous users (optional keys user_zeta, user_kappa, user_p_tx,
    user_local_freq, Sec. II): user m's latency is zeta_m * work / f with its
    own levels, its energy kappa_m * work * f^2, its upload energy p_m * up;
    the gamma order (Eq. (17)) is then taken per partition point.
    """
    mode = int(prob.get("mode", 0))
    N, L, K, J = prob["N"], prob["L"], prob["K"], prob["J"]
    cyc = [_F(x) for x in prob["cycles"][inst]]
    bits = [_F(x) for x in prob["bits"][inst]]
    al = [_F(x) for x in prob["alpha"][inst]]
    be = [_F(x) for x in prob["beta"][inst]]
    rate = [_F(x) for x in prob["rate"][inst]]
    T = [_F(x) for x in prob["deadline"][inst]]
    tfree = _F(prob["t_free"][inst]) if prob.get("t_free") is not None else Fraction(0)
    g = [_F(x) for x in prob["gpu_freq"]]
    gc, p0 = _F(prob["gpu_c"]), _F(prob["gpu_p_static"])

    def per_user(key, shared):
        a = prob.get(key)
        return [_F(a[inst][m]) for m in range(N)] if a is not None else [shared] * N

    zeta = per_user("user_zeta", Fraction(1))
    kap = per_user("user_kappa", _F(prob["kappa"]))
    ptxm = per_user("user_p_tx", _F(prob["p_tx"]))
    if prob.get("user_local_freq") is not None:
        fu = [[_F(x) for x in prob["user_local_freq"][inst][m]] for m in range(N)]
    else:
        fu = [[_F(x) for x in prob["local_freq"]]] * N

    def local_t(m, s, k):   # Eq. (1), layers 1..s, user m
        return sum((zeta[m] * c / fu[m][k] for c in cyc[:s]), Fraction(0))

    def local_e(m, s, k):   # Eq. (2), layers 1..s, user m
        return sum((kap[m] * c * fu[m][k] * fu[m][k] for c in cyc[:s]), Fraction(0))

    def upload(m, s):    # Eq. (3)
        return bits[s] / rate[m]

    def gpu_t(s, j, b):  # Eq. (5), layers s+1..L
        return sum(((al[l] + be[l] * b) * g[J - 1] / g[j] for l in range(s, L)), Fraction(0))

    best = None   # (energy, order key, policy)
    energies = []

    cont = bool(mode & MODE_CONTINUOUS)

    def cycles(s):
        return sum(cyc[:s], Fraction(0))

    def cont_choice(m, s, budget):
        """(frequency, energy, latency) of user m's slowest frequency
        finishing layers 1..s within budget, or None."""
        c = cycles(s)
        fmin, fmax = fu[m][0], fu[m][K - 1]
        if c == 0:   # nothing to compute: (7) still needs the upload in time
            return (fmin, Fraction(0), Fraction(0)) if budget >= 0 else None
        w = zeta[m] * c
        if budget <= 0 or w / budget > fmax:
            return None
        fr = max(fmin, w / budget)
        return fr, kap[m] * c * fr * fr, w / fr

    # local computing
    lc = None
    if cont:
        ch = [cont_choice(m, L, T[m]) for m in range(N)]
        if all(x is not None for x in ch):
            lc = (sum(x[1] for x in ch), tuple(x[0] for x in ch))
    else:
        for kv in product(range(K), repeat=N):
            if all(local_t(m, L, kv[m]) <= T[m] for m in range(N)):
                E = sum(local_e(m, L, kv[m]) for m in range(N))
                if lc is None or E < lc[0]:
                    lc = (E, kv)

    def try_set(s, j, S):
        """Best level vector for offloading set S at (s, j), or None."""
        b = len(S)
        lo = min(T[m] for m in S)                                 # Eq. (10)
        phi = gpu_t(s, j, b)
        if not (tfree + phi <= lo):                               # (6)
            return None
        P = gc * g[j] ** 3 + p0
        if cont:
            E, ready, kv = P * phi, tfree, []
            for m in range(N):
                if m in S:
                    x = cont_choice(m, s, lo - phi - upload(m, s))             # (7), Eq. (20)
                    if x is None:
                        return None
                    E += x[1] + ptxm[m] * upload(m, s)
                    ready = max(ready, x[2] + upload(m, s))
                else:
                    x = cont_choice(m, L, T[m])                                # (8)
                    if x is None:
                        return None
                    E += x[1]
                kv.append(x[0])
            return E, dict(cut=s, gpu_level=j, batch=b, levels=tuple(kv),
                           offload=tuple(int(m in S) for m in range(N)),
                           t_free_out=ready + phi)                            # Eq. (22)
        choice = None
        for kv in product(range(K), repeat=N):
            ok = True
            E = P * phi
            for m in range(N):
                if m in S:
                    ok = ok and local_t(m, s, kv[m]) + upload(m, s) + phi <= lo   # (7)
                    E += local_e(m, s, kv[m]) + ptxm[m] * upload(m, s)
                else:
                    ok = ok and local_t(m, L, kv[m]) <= T[m]                     # (8)
                    E += local_e(m, L, kv[m])
                if not ok:
                    break
            if ok and (choice is None or E < choice[0]):
                choice = (E, kv)
        if choice is None:
            return None
        E, kv = choice
        ready = max([tfree] + [local_t(m, s, kv[m]) + upload(m, s) for m in S])
        return E, dict(cut=s, gpu_level=j, batch=b, levels=kv,
                       offload=tuple(int(m in S) for m in range(N)),
                       t_free_out=ready + phi)                    # Eq. (22)

    def threshold(s, lst, i):
        """Eq. (18) for the i-th user (1-based) of lst: the lowest f_e at
        which the suffix lst[i:B] can batch; None if no f_e is enough (a
        non-positive denominator)."""
        S = lst[i - 1:]
        phi = gpu_t(s, J - 1, len(S)) * g[J - 1]   # latency times frequency
        h = lst[i - 1]
        den = min(T[m] for m in S) - (upload(h, s) + local_t(h, s, K - 1))   # Eq. (17)
        return phi / den if den > 0 else None

    s_end = 1 if mode & MODE_BINARY else L
    j_low = J - 1 if mode & MODE_FIXED_EDGE else 0
    for s in range(s_end):
        # Alg. 1 offloads the tail of the gamma-descending list (Eq. (17)):
        # the b smallest gamma; equal gamma offloads the lower index first
        order = sorted(range(N), key=lambda m: (upload(m, s) + local_t(m, s, K - 1), m))
        if mode & MODE_GREEDY:
            lst = order[::-1]                     # list(M'), gamma descending
            fth = [threshold(s, lst, i) for i in range(1, N + 1)]
            ihat = next((i for i in range(1, N + 1) if fth[i - 1] is not None), N + 1)
            for j in range(J - 1, j_low - 1, -1):
                while ihat <= N and (fth[ihat - 1] is None or g[j] < fth[ihat - 1]):
                    ihat += 1                     # the head leaves the batch
                if ihat > N:
                    break                         # empty set ends the sweep
                got = try_set(s, j, lst[ihat - 1:])
                if got is not None:
                    energies.append(got[0])
                    if best is None or got[0] < best[0]:
                        best = got
            continue
        for j in range(J - 1, j_low - 1, -1):
            for mask in range((1 << N) - 1, 0, -1):
                S = [m for m in range(N) if (mask >> m) & 1]
                b = len(S)
                if suffix_only and set(S) != set(order[:b]):
                    continue
                got = try_set(s, j, S)
                if got is None:
                    continue
                energies.append(got[0])
                if best is None or got[0] < best[0]:
                    best = got
    if lc is not None:
        energies.append(lc[0])
        if best is None or lc[0] < best[0]:
            best = (lc[0], dict(cut=L, gpu_level=-1, batch=0, levels=lc[1],
                                offload=(0,) * N, t_free_out=tfree))
    if best is None:
        return None
    E, pol = best
    rest = sorted(energies)
    pol["energy"] = E
    pol["energy_second"] = rest[1] if len(rest) > 1 else None
    return pol


FRONT = 16  # states kept per prefix (JO_FRONT of the oracle)


def front_add(front, state):
    """Adds state (E, T, ...) to a front sorted by energy: nothing happens if
    a kept state has no higher energy and no later release (it came first);
    otherwise the states it dominates leave, it enters at its energy's
    place, and a front longer than FRONT loses its highest energy."""
    E, T = state[0], state[1]
    if any(f[0] <= E and f[1] <= T for f in front):
        return front
    kept = [f for f in front if not (E <= f[0] and T <= f[1])]
    at = len(kept)
    while at > 0 and kept[at - 1][0] > E:
        at -= 1
    kept.insert(at, state)
    return kept[:FRONT]


def solve_grouped_exact(prob, inst):
    """Outer grouping of one instance in exact arithmetic: users sorted by
    deadline (ties by index), consecutive groups served in that order, each
    group solved by solve_exact on its own users (in user index order) with
    the GPU free at the previous group's release time.  For every prefix i
    of the order the program keeps a front of (energy, release) states that
    no other state dominates (no higher energy and no later release), built
    in the order j = 0..i-1, then the states of the front of j from the
    earliest release to the latest; the answer is the lowest-energy state of
    the full order.  Returns None if no
    grouping is feasible, else dict(energy, t_free_out, ends, groups)."""
    N = prob["N"]
    T = [_F(x) for x in prob["deadline"][inst]]
    order = sorted(range(N), key=lambda m: (T[m], m))
    t0 = _F(prob["t_free"][inst]) if prob.get("t_free") is not None else Fraction(0)

    def group_solve(a, b, tfree):
        members = sorted(order[a:b])
        sub = {k: prob[k] for k in ("local_freq", "gpu_freq", "kappa", "p_tx", "gpu_c",
                                     "gpu_p_static", "K", "J", "L", "dtype")}
        sub["mode"] = prob.get("mode", 0)
        sub["N"] = len(members)
        for k in ("cycles", "bits", "alpha", "beta"):
            sub[k] = prob[k][inst:inst + 1]
        sub["rate"] = prob["rate"][inst:inst + 1, members]
        sub["deadline"] = prob["deadline"][inst:inst + 1, members]
        for k in ("user_zeta", "user_kappa", "user_p_tx", "user_local_freq"):
            if prob.get(k) is not None:   # heterogeneous users: the members' own
                sub[k] = prob[k][inst:inst + 1, members]
        sub["t_free"] = [tfree]
        return solve_exact(sub, 0, suffix_only=True)

    # front[i]: states (energy, release, end, previous state, group policy)
    fronts = {0: [(Fraction(0), t0, 0, None, None)]}
    for i in range(1, N + 1):
        front = []
        for j in range(i):
            for st in reversed(fronts.get(j, [])):  # the earliest release first
                pol = group_solve(j, i, st[1])
                if pol is not None:
                    front = front_add(front, (st[0] + pol["energy"], pol["t_free_out"], i, st, pol))
        if front:
            fronts[i] = front
    if N not in fronts:
        return None
    best = fronts[N][0]
    ends, groups, st = [], [], best
    while st[3] is not None:
        ends.append(st[2])
        groups.append(st[4])
        st = st[3]
    return dict(energy=best[0], t_free_out=best[1], ends=ends[::-1], groups=groups[::-1])


def user_tables_exact(prob, inst):
    """Stage-1 tables of one instance (users sharing their parameters) in
    exact arithmetic, from the system model of Sec. II:

    up[s][m]     = O_s / R_m for s < L, 0 for s = L (nothing is uploaded),
                   Eq. (3);
    t[s][k]      = C[s] / f_k, C[s] the cycles of layers 1..s, Eq. (1);
    gamma[s][m]  = up[s][m] + t[s][K-1], the minimum latency cost, Eq. (17);
    level[s][m]  = the lowest k with t[s][k] <= T_m - up[s][m] (Eq. (20) on
                   the levels against the user's own deadline), None if no
                   level fits;
    energy[s][m] = kappa f_k^2 C[s] + p_tx up[s][m] at that level, Eqs. (2),
                   (4) (None if no level);
    slack[s][m]  = (T_m - up[s][m]) - t[s][k] at that level, at k = K-1 if
                   none fits;
    margin[s][m] = min over k of |t[s][k] - (T_m - up[s][m])|: how far the
                   level decision is from a tie.
    Also the rate order pi (rate descending, ties to the lower index), the
    batch deadlines lo[b] (Eq. (10)) and bmin."""
    N, L, K = prob["N"], prob["L"], prob["K"]
    cyc = [_F(x) for x in prob["cycles"][inst]]
    bits = [_F(x) for x in prob["bits"][inst]]
    rate = [_F(x) for x in prob["rate"][inst]]
    T = [_F(x) for x in prob["deadline"][inst]]
    f = [_F(x) for x in prob["local_freq"]]
    kappa, ptx = _F(prob["kappa"]), _F(prob["p_tx"])
    rows = {k: [[None] * N for _ in range(L + 1)]
            for k in ("up", "gamma", "level", "energy", "slack", "margin", "t_top")}
    for s in range(L + 1):
        C = sum(cyc[:s], Fraction(0))
        t = [C / fk for fk in f]
        for m in range(N):
            up = bits[s] / rate[m] if s < L else Fraction(0)
            budget = T[m] - up
            lv = next((k for k in range(K) if t[k] <= budget), None)
            kk = lv if lv is not None else K - 1
            rows["up"][s][m] = up
            rows["gamma"][s][m] = up + t[K - 1]
            rows["level"][s][m] = lv
            rows["energy"][s][m] = None if lv is None else kappa * f[lv] * f[lv] * C + ptx * up
            rows["slack"][s][m] = budget - t[kk]
            rows["margin"][s][m] = min(abs(tk - budget) for tk in t)
            rows["t_top"][s][m] = t[K - 1]
    pi = sorted(range(N), key=lambda m: (-rate[m], m))
    lo = [min(T[m] for m in pi[:b]) for b in range(1, N + 1)]
    bad = [i for i in range(N) if rows["level"][L][pi[i]] is None]
    rows.update(order=pi, batch_deadline=lo, min_batch=(bad[-1] + 1) if bad else 0)
    return rows
