// placement.h -- workgroup -> work-item map for the two placement modes.
//
// Shared by the device kernels and the host (which fills the kernel-argument
// view and mirrors the map for inspection).
//
// Work items are numbered group-major: item = group * group_size + member.
// A logical group is the set of work items that touch the same input chunk
// (Sec. 4.2.1: a threadblock joins the group it shares chunks with, and
// Algorithm 1 places each group as a unit).  Groups may also have variable
// sizes (all-to-all); the host then lists the items in placement order.
//
// MI355X dispatches workgroup b of a launch to XCD (b mod 8).  With G
// workgroups, XCD x holds Gx = ceil((G - x) / 8) of them; its k-th one has
// k = b div 8.
//
//  LINEAR (UA, Sec. 5.3): workgroup b runs items b, b+G, b+2G, ...  The
//      members of a group (consecutive items) are spread over different XCDs.
//
//  XCD (NAP*, Sec. 5.3): Algorithm 1 hands logical groups round-robin to the
//      domains (the next domain for each group) and keeps every group inside
//      one domain.  Here the domains are the 8 XCDs: group g goes to XCD
//      g mod 8, and XCD x runs its groups x, x+8, x+16, ... member by member
//      on consecutive workgroups, so the members of a group run at the same
//      time on one XCD and re-read their shared chunk from that XCD's L2.
//      A group of one item is placed exactly as LINEAR places it.
#pragma once

#include <stdint.h>

#ifndef NUNA_HD
#if defined(__HIPCC__)
#define NUNA_HD __host__ __device__
#else
#define NUNA_HD
#endif
#endif

namespace nuna {

constexpr int kNumXcd = 8;
constexpr int kPlaceLinear = 0;
constexpr int kPlaceXcd = 1;

struct ItemRange {
    int64_t first;
    int64_t end;
    int64_t stride;
};

// Kernel-argument view of a placement.
//  Uniform groups (gsize > 0): `groups` groups of gsize items each.
//  Listed order (gsize == 0): the items are already stored in placement
//      order; XCD x runs list positions [start[x], start[x+1]).
struct Place {
    int64_t groups;
    int64_t start[kNumXcd + 1];
    int32_t mode;
    int32_t gsize;
    int32_t gshift;  // log2(gsize) when a power of two, else -1
    int32_t pad;
};

NUNA_HD inline int64_t place_items(const Place& pl) {
    return pl.gsize > 0 ? pl.groups * pl.gsize : pl.start[kNumXcd];
}

// The linear map runs when:
//  - the mode is LINEAR;
//  - groups have one item each: dealing single items round-robin to the XCDs
//    is exactly what LINEAR does, so the same code runs;
//  - the launch has fewer than 8 workgroups and cannot reach every XCD.
NUNA_HD inline bool linear_map(const Place& pl, int64_t G) {
    return pl.mode == kPlaceLinear || pl.gsize == 1 || G < kNumXcd;
}

// Range of list positions workgroup b of G runs under per-XCD item lists
// (gsize 0): with the linear map, every b-th position of all `total`;
// otherwise XCD x = b mod 8 runs its list [start_x, start_x1), its
// workgroups taking every (workgroups on x)-th position.
NUNA_HD inline ItemRange list_items(bool linear, int64_t start_x, int64_t start_x1, int64_t total, int64_t b,
                                    int64_t G) {
    ItemRange r;
    if (linear) {
        r.first = b;
        r.end = total;
        r.stride = G;
        return r;
    }
    const int64_t x = b & (kNumXcd - 1);
    r.first = start_x + (b >> 3);
    r.end = start_x1;
    r.stride = (G - x + kNumXcd - 1) >> 3;
    return r;
}

// Range of list positions workgroup b of G runs.
NUNA_HD inline ItemRange items_of(const Place& pl, int64_t b, int64_t G) {
    const int64_t x = b & (kNumXcd - 1);
    if (pl.gsize == 0) return list_items(linear_map(pl, G), pl.start[x], pl.start[x + 1], pl.start[kNumXcd], b, G);
    ItemRange r;
    if (linear_map(pl, G)) {
        r.first = b;
        r.end = place_items(pl);
        r.stride = G;
        return r;
    }
    const int64_t gx = pl.groups > x ? (pl.groups - x + kNumXcd - 1) >> 3 : 0;
    r.first = b >> 3;
    r.end = gx * pl.gsize;
    r.stride = (G - x + kNumXcd - 1) >> 3;
    return r;
}

// Work item at list position i of workgroup b of G.
NUNA_HD inline int64_t item_at(const Place& pl, int64_t b, int64_t G, int64_t i) {
    if (linear_map(pl, G) || pl.gsize == 0) return i;
    const int64_t x = b & (kNumXcd - 1);
    int64_t q, m;
    if (pl.gshift >= 0) {
        q = i >> pl.gshift;
        m = i & ((int64_t(1) << pl.gshift) - 1);
    } else {
        q = i / pl.gsize;
        m = i - q * pl.gsize;
    }
    return (x + kNumXcd * q) * pl.gsize + m;
}

inline int log2_exact(int64_t v) {
    for (int k = 0; k < 62; ++k)
        if ((int64_t(1) << k) == v) return k;
    return -1;
}

// Host: placement of `groups` uniform groups of `gsize` items.
inline Place make_place_uniform(int mode, int64_t groups, int64_t gsize) {
    Place pl{};
    pl.mode = mode;
    pl.groups = groups;
    pl.gsize = static_cast<int32_t>(gsize);
    pl.gshift = log2_exact(gsize);
    return pl;
}

// ---------------------------------------------------------------- page groups
//
// Launches that run one work item per workgroup (the direct kernels) number
// their items by address: item i covers bytes [i*cb, (i+1)*cb) of every rank
// buffer, cb the chunk bytes.  When a chunk is smaller than a 4 KiB page
// (Sec. 4.2 places memory in 4 kB pages), the gp = 4096 / cb items of one
// page touch the same page of every buffer: in XCD mode they form one logical
// group (Sec. 4.2.1), and groups are dealt round-robin to the XCDs with their
// members on consecutive slots of one XCD (as in Algorithm 1), so no page's
// work is split between XCDs.  LINEAR runs item b on workgroup b, which puts
// the gp items of a page on gp different XCDs.
//
// gshift = log2(gp) (0: the linear map).  Workgroup b = 8k + x runs item
// (8 * (k >> gshift) + x) << gshift | (k mod gp); the grid is padded to whole
// rounds of 8 groups, and workgroups past the last item exit.
NUNA_HD inline int64_t page_item(int64_t b, int gshift) {
    if (gshift == 0) return b;
    const int64_t x = b & (kNumXcd - 1);
    const int64_t k = b >> 3;
    const int64_t q = k >> gshift;
    const int64_t m = k & ((int64_t(1) << gshift) - 1);
    return ((q << 3) + x) << gshift | m;
}

// Host: workgroups of a page-grouped launch over `items` work items.
inline int64_t page_grid(int64_t items, int gshift) {
    if (gshift == 0) return items;
    const int64_t gp = int64_t(1) << gshift;
    const int64_t groups = (items + gp - 1) / gp;
    return kNumXcd * ((groups + kNumXcd - 1) / kNumXcd) * gp;
}

// Host: log2 of the items per page for chunks of `chunk_bytes` (a power of
// two times 16), 0 when a chunk covers a whole page or more.
inline int page_shift(int64_t chunk_bytes) {
    int s = 0;
    while ((chunk_bytes << (s + 1)) <= 4096) ++s;
    return s;
}

// Host: workgroups a launch of this placement needs so that every item gets
// its own workgroup (before any cap).  XCD mode sizes every XCD for the
// largest per-XCD group list; workgroups past a list's end exit at once.
inline int64_t place_grid(const Place& pl) {
    if (pl.mode == kPlaceLinear || pl.gsize <= 1) return place_items(pl);
    return kNumXcd * ((pl.groups + kNumXcd - 1) / kNumXcd) * pl.gsize;
}

}  // namespace nuna
