"""ORACLE - test infrastructure only: the heterogeneous module scheduler.

HeteGen Sec. 4.5 "Heterogeneous Module Scheduler": when GPU memory is left over,
whole modules are moved onto the GPU.  The benefit of moving one module is the time
it saves per unit of GPU memory it takes, Eq. 13: g = T_CPU / Mem, where T_CPU is
the module's benchmarked heterogeneous time (the balanced time of Eq. 11, which the
module no longer costs once its weights are resident) and Mem the bytes its resident
copy takes.  Modules are moved in order of decreasing g, layer by layer, until the
GPU memory limit is reached.

Readings (the paper leaves them open, Fig. 7 is not available):
- "for each layer" is a round robin over the layers: every layer's highest-g module
  first (layers in index order), then every layer's second-highest, and so on;
  equal g within a layer keeps the modules' index order;
- a module that does not fit in the memory still free is skipped and the walk goes
  on, so a later, smaller module can still take the rest of the budget;
- a resident module is computed wholly on the GPU (CPU fraction 0).
"""


def gains(t_cpu, mem):
    """Eq. 13 for every module."""
    return [t / m for t, m in zip(t_cpu, mem)]


def visit_order(t_cpu, mem, layer):
    """Module indices in the order the scheduler considers them."""
    g = gains(t_cpu, mem)
    by_layer = {}
    for i, l in enumerate(layer):
        by_layer.setdefault(l, []).append(i)
    ranked = {}
    for l, mods in by_layer.items():
        # decreasing g; a stable sort keeps index order among equal gains
        ranked[l] = sorted(mods, key=lambda i: -g[i])
    order = []
    depth = max(len(v) for v in ranked.values()) if ranked else 0
    for r in range(depth):
        for l in sorted(ranked):
            if r < len(ranked[l]):
                order.append(ranked[l][r])
    return order


def schedule(t_cpu, mem, layer, budget):
    """Resident flag per module and the bytes they take."""
    resident = [0] * len(t_cpu)
    used = 0.0
    for i in visit_order(t_cpu, mem, layer):
        if used + mem[i] <= budget:
            resident[i] = 1
            used += mem[i]
    return resident, used
