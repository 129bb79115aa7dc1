"""Oracle: the mixed-precision bit allocation of Section 3.3.  TEST INFRASTRUCTURE ONLY.

What it follows (Section 3.3, "Tensor-Level Sensitivity Analysis",
"Hardware-Constrained Budget Formulation" and "Dynamic Allocation with
Back-off"):

* Sens(t) = (PPL(Q_low) - PPL(Q_high, t)) / rho_t with rho_t = |t| / |layer(t)|;
* S_low = P_pruned * b(Q_low) / (8 * 10^9) GB, B_base = M_limit - S_low;
* lowering a tensor from Q_low to Q_low' releases
  B_delta = |t| * (b(Q_low, t) - b(Q_low', t)) / (8 * 10^9), and
  B_total = B_base + (the releases so far);
* tensors in descending Sens order are upgraded: fewer than 10M parameters
  to Q8, 10M to 50M to Q6; routed experts are never upgraded; the upgrades
  must satisfy  sum_{t in T_up} |t| (b(Q_new, t) - b(Q_low, t)) / (8 * 10^9) <= B_total;
* back-off when an upgrade does not fit: (1) the current tensor one level,
  then two levels lower; (2) the largest previously upgraded tensor one
  level lower, never below Q4; (3) routed experts from Q_low to Q_low', in
  binary-partition layer order, gate and up projections before the others.

Readings where the paper is silent or loose (listed with the design notes):

* widths are bits per weight (scales included) in units of 1/64 bit and
  sizes are integers of such units, so every fit decision is exact; GB
  figures are those integers divided by 64 * 8 * 10^9;
* every tensor starts at Q_low (the paper's single b(Q_low));
* the ladder of widths is given: index low' < low < floor (Q4) <= Q6 <= Q8;
  "one level" is one step on the ladder (Q8 -> Q6 when no Q7 exists);
* tensors above 50M parameters that are not routed experts are not
  upgraded (the paper states no tier for them);
* rule 1 tries the target, then one, then two levels lower, never below
  the floor; if none fits, rules 2 and 3 free memory until the tensor fits
  at the lowest level rule 1 tried;
* rules 2 and 3 run only when together they can free enough for the
  current tensor; otherwise it stays at Q_low and nothing is downgraded for
  it;
* rule 2's "most parameters": ties go to the tensor later in the Sens order;
* rule 3's order: the binary partition of the MoE layer positions 0..L-1,
  breadth first over half-open intervals [lo, hi) with midpoint
  ceil((lo + hi) / 2) (this reproduces the printed 29, 15, 44, 8 for 58
  layers); first the gate then the up tensors of each layer in that order,
  then the down tensors in the same layer order; ties by tensor index;
* if even Q_low does not fit (B_base < 0), rule 3 runs before any upgrade;
  the plan is infeasible if it cannot release enough;
* Sens ties: lower tensor index first.
"""
from collections import deque

OTHER, ROUTED_GATE, ROUTED_UP, ROUTED_DOWN = 0, 1, 2, 3
BITS_PER_GB = 8 * 10 ** 9
UNITS_PER_BIT = 64


def sensitivity(ppl_low, ppl_high, params, layer_params):
    """Sens(t) for every tensor (float64)."""
    out = []
    for ph, p, lp in zip(ppl_high, params, layer_params):
        rho = float(p) / float(lp)
        out.append((float(ppl_low) - float(ph)) / rho)
    return out


def binary_partition_order(n_layers):
    """MoE layer positions 0..n_layers-1 in binary-partition order."""
    order, queue = [], deque([(0, n_layers)])
    while queue:
        lo, hi = queue.popleft()
        if lo >= hi:
            continue
        mid = (lo + hi + 1) // 2
        order.append(mid if mid < hi else hi - 1)
        m = order[-1]
        queue.append((lo, m))
        queue.append((m + 1, hi))
    return order


def gb(units):
    return float(units) / float(UNITS_PER_BIT * BITS_PER_GB)


def plan_bits(params, sens, kind, layer, *, ladder, low_prime, low, floor, small_level, medium_level,
              m_limit_bytes, n_moe_layers, small_params=10_000_000, medium_params=50_000_000):
    """-> (levels list, report dict).  ladder: widths in 1/64 bit, ascending."""
    n = len(params)
    level = [low] * n
    T_up = []                                   # upgraded tensors, in upgrade order

    def size(t, lv):
        return params[t] * ladder[lv]

    def used():
        return sum(size(t, level[t]) - size(t, low) for t in T_up)

    S_low = sum(size(t, low) for t in range(n))
    B_base = m_limit_bytes * 8 * UNITS_PER_BIT - S_low
    released = [0]

    def B_total():
        return B_base + released[0]

    # rule 3's queue: gate/up of each layer in partition order, then down
    part = binary_partition_order(n_moe_layers)
    routed_queue = deque()
    for L in part:
        for k in (ROUTED_GATE, ROUTED_UP):
            routed_queue.extend(t for t in range(n) if kind[t] == k and layer[t] == L)
    for L in part:
        routed_queue.extend(t for t in range(n) if kind[t] == ROUTED_DOWN and layer[t] == L)
    n_rule3 = [0]

    def rule3():
        if not routed_queue:
            return False
        t = routed_queue.popleft()
        released[0] += size(t, low) - size(t, low_prime)
        level[t] = low_prime
        n_rule3[0] += 1
        return True

    while used() > B_total():
        if not rule3():
            break

    def tier(t):
        if kind[t] != OTHER:
            return None
        if params[t] < small_params:
            return small_level
        if params[t] <= medium_params:
            return medium_level
        return None

    by_sens = sorted((t for t in range(n) if tier(t) is not None), key=lambda t: (-sens[t], t))
    rank = {t: i for i, t in enumerate(by_sens)}
    n_rule2 = 0
    for t in by_sens:
        target = tier(t)
        tries = [lv for lv in (target, target - 1, target - 2) if lv >= floor]
        placed = False
        for lv in tries:                                          # rule 1
            if used() + size(t, lv) - size(t, low) <= B_total():
                level[t] = lv
                T_up.append(t)
                placed = True
                break
        if placed:
            continue
        lv = tries[-1]
        can_free = (sum(size(u, level[u]) - size(u, floor) for u in T_up)
                    + sum(size(q, low) - size(q, low_prime) for q in routed_queue))
        if used() + size(t, lv) - size(t, low) - B_total() > can_free:
            continue                                              # stays at Q_low
        while used() + size(t, lv) - size(t, low) > B_total():
            above = [u for u in T_up if level[u] > floor]
            if above:                                             # rule 2
                u = max(above, key=lambda u: (params[u], rank[u]))
                level[u] -= 1
                n_rule2 += 1
            else:
                rule3()                                           # rule 3
        level[t] = lv
        T_up.append(t)

    u = used()
    report = dict(S_low=S_low, B_base=B_base, B_delta=released[0], B_total=B_total(), used=u,
                  total=S_low - released[0] + u, n_upgraded=len(T_up), n_rule2=n_rule2,
                  n_rule3=n_rule3[0], feasible=u <= B_total())
    return level, report
