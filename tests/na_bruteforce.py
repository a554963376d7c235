"""Pure-Python brute-force neighbourhoods, written independently of the oracle.

Along each axis a query keeps the k nearest coordinates of its own dilation
group (the sub-lattice x = g mod d, Sec. 3.4), ranking candidates by distance
and taking the lower coordinate among equally near ones; the neighbourhood of
a multi-axis query is the product of its per-axis sets (the attention weights
of a T_h x T_w query tile have shape T_h x T_w x k_h k_w, Sec. 3.2).  There is
no window-start formula here: only "nearest", as the paper words it (Sec. 1,
Sec. 2).  Along a causal axis (Sec. 3.4, Fig. "neighborhoodattention"
caption) only coordinates not larger than the query's are candidates.
"""
import itertools


def axis_neighbours(x, length, k, d, causal=False):
    group = [j for j in range(length) if j % d == x % d and (not causal or j <= x)]
    ranked = sorted(group, key=lambda j: (abs(j - x), j))
    return sorted(ranked[:k])


def neighbours(extents, kernel_size, dilation, causal=None):
    """List over flat tokens (row-major, axis 0 outermost) of sorted flat neighbour indices."""
    rank = len(extents)
    causal = causal or [False] * rank
    coords = list(itertools.product(*[range(e) for e in extents]))
    strides = [1] * rank
    for a in range(rank - 2, -1, -1):
        strides[a] = strides[a + 1] * extents[a + 1]
    result = []
    for c in coords:
        per_axis = [axis_neighbours(c[a], extents[a], kernel_size[a], dilation[a], causal[a])
                    for a in range(rank)]
        flat = sorted(sum(j * s for j, s in zip(combo, strides)) for combo in itertools.product(*per_axis))
        result.append(flat)
    return result


def read_golden_windows(path):
    """Parse tests/golden/windows_1d.txt into {(L, k, d): {x: [neighbours]}}."""
    blocks = {}
    cur = None
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("L="):
                parts = dict(p.split("=") for p in line.split())
                cur = (int(parts["L"]), int(parts["k"]), int(parts["d"]))
                blocks[cur] = {}
            else:
                x, rest = line.split(":")
                blocks[cur][int(x)] = [int(t) for t in rest.split()]
    return blocks
