"""LDS bank-conflict model of the matrix-core kernel on gfx950, and what it
says about the kernel's LDS layouts.

The model was fitted to `rocprofv3 --pmc SQ_LDS_BANK_CONFLICT SQ_INSTS_LDS`
runs of a probe kernel that reads LDS at chosen per-lane addresses
(`bench.py --lds-probe`, kernel `lds_probe` in bench_peaks.hip); the measured
table is profiles/lds_bank_probe.json.  It reproduces every 4- and 8-byte
pattern measured:

* ds_read_b32: 32 banks of 4 bytes; a wave64 read is served as two
  half-waves of 32 lanes (lanes 0-31, 32-63); within a half, lanes reading
  the same word are served together, and the read takes one extra pass per
  further distinct word that falls in the same bank.  SQ_LDS_BANK_CONFLICT
  counts those extra passes, summed over both halves.
* ds_read_b64: the same with 64 banks of 4 bytes (a lane's two words in
  consecutive banks).
* ds_read_b128 follows neither rule; its measured costs are used as they
  are.  Lane (g, l) at word A*l + B*g with A = 12 or 28 (a 3x3 or 5x5 tap
  run padded to a multiple of 4) and B a multiple of 64 measured 0: the
  weights-through-LDS layout of the kernel is that.

The implicit-GEMM kernel's B operand (the input halo) is read with
ds_read_b32: lane (g, l) of a 16x16x4 step reads channel plane g (offset
g*PL words; g*G4*PL for the 1x1 variants whose lanes take consecutive
channels, `lstep` = G4) at tile pixel p = 16n + l of its block n (row p / TW,
column p % TW, so word (p / TW)*S*HCP + (p % TW)*S within the plane); tap and
channel-group offsets shift every lane alike and do not change the cost.
`b_read_costs` gives the cost of each block's read for a layout (row pitch
HCP, plane pitch PL), `best_halo_layout` the smallest conflict-free layout.
Measured on MI355X, the kernel is faster with its halo stored unpadded
(HCP = HC, PL = HR*HC, at most two extra passes per read) than with the
conflict-free padded layouts: the padding is halo DMA the small-tile
kernels wait on, while a conflict adds a pass to a read issued steps ahead.

    python -m paper_1909_02765_amd.lds_banks     # costs of the kernel's layouts
"""
from __future__ import annotations

def conflicts_b32(addrs):
    """Extra passes of one ds_read_b32 at word addresses addrs[0..63]."""
    tot = 0
    for h in (0, 32):
        banks = {}
        for a in addrs[h:h + 32]:
            banks.setdefault(a % 32, set()).add(a)
        tot += max(len(v) for v in banks.values()) - 1
    return tot


def conflicts_b64(addrs):
    """Extra passes of one ds_read_b64 at word addresses addrs[0..63] (even)."""
    tot = 0
    for h in (0, 32):
        banks = {}
        for a in addrs[h:h + 32]:
            for k in (0, 1):
                banks.setdefault((a + k) % 64, set()).add(a + k)
        tot += max(len(v) for v in banks.values()) - 1
    return tot


def b_read_addresses(TH, TW, S, HCP, PL, NWP, wp, n, lstep=1):
    """Word addresses of the B read of pixel block n of wave group wp, lanes 0..63
    (the tail block of a 16q + t pixel tile, t <= 4, reads t pixels, lanes
    16kq + 4cg + j on pixel j; lanes past the tile read pixel 0)."""
    npix = TH * TW
    nb = (npix + 16 * NWP - 1) // (16 * NWP)
    tailp = npix % 16
    tail4 = NWP == 1 and 1 <= tailp <= 4
    out = []
    for lane in range(64):
        g, l = lane >> 4, lane & 15
        p = (wp * nb + n) * 16 + ((l & 3) if (tail4 and n == nb - 1) else l)
        if p >= npix:
            p = 0
        out.append(g * lstep * PL + (p // TW) * S * HCP + (p % TW) * S)
    return out


def b_read_costs(TH, TW, S, HCP, PL, NWP=1, lstep=1):
    npix = TH * TW
    nb = (npix + 16 * NWP - 1) // (16 * NWP)
    return [conflicts_b32(b_read_addresses(TH, TW, S, HCP, PL, NWP, wp, n, lstep))
            for wp in range(NWP) for n in range(nb)]


def tight_layout(TH, TW, S, K):
    """The kernel's layout for halos other than the 16x16 one: unpadded."""
    hr, hc = (TH - 1) * S + K, (TW - 1) * S + K
    return hc, hr * hc


def rule_of_thumb_layout(TH, TW, S, K):
    """The kernel's earlier layout rule (row pitch chosen so that successive
    planes fall on opposite bank halves), kept for comparison."""
    hr, hc = (TH - 1) * S + K, (TW - 1) * S + K
    for r in range(hc, hc + 64):
        if S % 2 == 1 and (hr * r) % 32 == 16:
            return r, hr * r
        if S % 2 == 0 and (hr * r) % 2 == 1:
            return r, hr * r
    return hc, hr * hc


def best_halo_layout(TH, TW, S, K, NWP=1):
    """(HCP, PL, conflict passes per read) minimising first the conflicts, then
    the plane size: HCP in [HC, HC + 32), PL in [HR*HCP, HR*HCP + 32)."""
    hr, hc = (TH - 1) * S + K, (TW - 1) * S + K
    best = None
    for hcp in range(hc, hc + 32):
        for pl in range(hr * hcp, hr * hcp + 32):
            costs = b_read_costs(TH, TW, S, hcp, pl, NWP)
            key = (sum(costs), pl, hcp)
            if best is None or key < best[0]:
                best = (key, hcp, pl, sum(costs) / len(costs))
    return best[1], best[2], best[3]


# Tile shapes (TH, TW, stride, K, NWP) of the compiled variants other than the
# 14x14 / 3x3 / stride-1 one (whose 16x16 halo keeps 16-word rows).
TILE_SHAPES = [(4, 4, 1, 1, 1), (4, 4, 1, 3, 1), (4, 4, 1, 5, 1), (4, 4, 2, 3, 1), (7, 7, 1, 1, 1),
               (7, 7, 1, 3, 1), (7, 7, 1, 5, 1), (7, 7, 2, 3, 1), (8, 8, 1, 3, 1), (8, 8, 1, 5, 1),
               (14, 14, 1, 1, 1), (8, 32, 1, 3, 2)]

def probe_patterns():
    """(name, dwords per lane, word address per lane) for the LDS probe."""
    L = range(64)
    P = []
    for st in (1, 2, 4, 16, 32, 64):
        P.append((f"b32_stride{st}", 1, [st * i for i in L]))
    P.append(("b32_same_word", 1, [0 for _ in L]))
    P.append(("b32_pairs_lane_mod32", 1, [i % 32 for i in L]))
    P.append(("b32_halves_64apart", 1, [(i % 32) + 64 * (i // 32) for i in L]))
    for gs in (16, 17, 144, 256, 272):
        P.append((f"b32_groups16_stride{gs}", 1, [(i % 16) + gs * (i // 16) for i in L]))
    for A in (2, 4, 6, 10, 34, 194):
        for B in (2, 16, 32):
            P.append((f"b64_l{A}_g{B}", 2, [A * (i % 16) + B * (i // 16) for i in L]))
    for A in (4, 8, 12, 16, 20, 28, 36, 196, 388):
        for B in (4, 12, 16, 64, 192, 256, 384, 448):
            P.append((f"b128_l{A}_g{B}", 4, [A * (i % 16) + B * (i // 16) for i in L]))
    for (th, tw, s, k, nwp) in TILE_SHAPES + [(14, 14, 1, 3, 1)]:
        for label, (hcp, pl) in (("rule", rule_of_thumb_layout(th, tw, s, k)),
                                 ("model", best_halo_layout(th, tw, s, k, nwp)[:2]),
                                 ("tight", tight_layout(th, tw, s, k))):
            if (th, tw, s, k) == (14, 14, 1, 3):
                hcp, pl = 16, 272
                if label != "rule":
                    continue
            npix = th * tw
            nb = (npix + 16 * nwp - 1) // (16 * nwp)
            for wp in range(nwp):
                for n in range(nb):
                    P.append((f"b32_tile{th}x{tw}_s{s}_k{k}_{label}_hcp{hcp}_pl{pl}_w{wp}_n{n}", 1,
                              b_read_addresses(th, tw, s, hcp, pl, nwp, wp, n)))
    return P


def model_cost(name, width, addrs):
    if width == 1:
        return conflicts_b32(addrs)
    if width == 2:
        return conflicts_b64(addrs)
    return None


def main():
    for (th, tw, s, k, nwp) in TILE_SHAPES:
        t = tight_layout(th, tw, s, k)
        tc = b_read_costs(th, tw, s, t[0], t[1], nwp)
        r = rule_of_thumb_layout(th, tw, s, k)
        rc = b_read_costs(th, tw, s, r[0], r[1], nwp)
        m = best_halo_layout(th, tw, s, k, nwp)
        print(f"tile {th}x{tw} s{s} k{k}: tight HCP {t[0]} PL {t[1]} -> {sum(tc) / len(tc):.2f} passes/read; "
              f"earlier rule HCP {r[0]} PL {r[1]} -> {sum(rc) / len(rc):.2f}; "
              f"conflict-free HCP {m[0]} PL {m[1]} -> {m[2]:.2f}")
    q = b_read_costs(14, 14, 1, 16, 272)
    print(f"tile 14x14 s1 k3 (16-word rows): HCP 16 PL 272 -> {sum(q) / len(q):.2f} passes/read")


if __name__ == "__main__":
    main()
