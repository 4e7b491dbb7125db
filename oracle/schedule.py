"""Launch order of the fused forward's 64-row query tiles, written out from
its definition (test infrastructure only; the product path never imports it).

The order is a permutation of the tiles t = (b*H + h) * ceil(L/64) + row/64:
first a stable sort by cost class descending, where a tile's cost is the
number of 64-key tiles its query block attends (list length times block/64)
and its class is 0 for no work, else bit_length(cost) capped at 15; then launch
slot s takes sorted position p(s), which hands each of the 8 XCDs runs of 256
consecutive positions: with G tiles and groups of 8*256 slots, for s inside
the whole groups p(s) = (s//8 // 256) * 2048 + (s % 8) * 256 + (s//8) % 256,
and p(s) = s for the slots of the last partial group.
"""
import numpy as np

XCDS = 8
RUN = 256


def cost_class(tiles: int) -> int:
    return 0 if tiles <= 0 else min(int(tiles).bit_length(), 15)


def launch_order(cnt, kmax: int, seqlen: int, block: int) -> np.ndarray:
    cnt = np.asarray(cnt)
    B, H, nb = cnt.shape
    ntiles = -(-seqlen // 64)
    spb = block // 64
    flat = cnt.reshape(-1)
    G = B * H * ntiles

    def cls(t):
        bh, qt = divmod(t, ntiles)
        c = int(min(max(flat[bh * nb + (qt * 64) // block], 0), kmax))
        return cost_class(c * spb)

    ordered = sorted(range(G), key=lambda t: (-cls(t), t))
    group = XCDS * RUN
    full = (G // group) * group
    out = np.empty(G, dtype=np.int32)
    for s in range(G):
        if s >= full:
            p = s
        else:
            r = s // XCDS
            p = (r // RUN) * group + (s % XCDS) * RUN + r % RUN
        out[s] = ordered[p]
    return out
