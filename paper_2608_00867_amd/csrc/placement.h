// placement.h -- workgroup -> work-item map for the two placement modes.
//
// Shared by the device kernels and the host (which precomputes the per-XCD
// table and mirrors the map for inspection).
//
// Work items are numbered group-major: item = group * group_size + member,
// where a logical group is the set of work items that touch the same input
// chunk (Sec. 4.2.1: threadblocks that share chunks are grouped, and a group
// is placed as a unit).  Groups may also have variable sizes (all-to-all);
// then the caller supplies the group start offsets.
//
// MI355X dispatches workgroup b of a launch to XCD (b mod 8).  With G
// workgroups, XCD x holds Gx = ceil((G - x) / 8) of them, and the XCDs before
// x hold S_x = sum_{x' < x} G_x' = a*x + min(x, c), where G = 8a + c.
//
//  LINEAR (UA, Sec. 5.3): workgroup b runs items b, b+G, b+2G, ...  With one
//      item per workgroup, consecutive items land on consecutive XCDs and the
//      members of a group are spread over different XCDs.
//
//  XCD (NAP*, Sec. 5.3): XCD x owns the contiguous item range
//      [start[x], start[x+1]), a share of the items proportional to its
//      workgroup count S_{x+1} - S_x, cut at group boundaries so no group is
//      split between XCDs (Algorithm 1 keeps a logical group inside one
//      domain).  Its k-th workgroup (k = b div 8) runs items start[x] + k,
//      start[x] + k + Gx, ...  Group members are consecutive items, so they run
//      concurrently on neighbouring workgroups of one XCD and share its L2.
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

// Kernel-argument view of a placement: for XCD mode start[0..8] are the
// per-XCD item ranges; for both modes start[8] is the total item count.
struct Place {
    int64_t start[kNumXcd + 1];
    int32_t mode;
    int32_t pad;
};

// Workgroups on XCDs 0..x-1 when G workgroups are dealt round-robin over 8 XCDs.
NUNA_HD inline int64_t wgs_before_xcd(int64_t x, int64_t G) {
    const int64_t a = G / kNumXcd, c = G % kNumXcd;
    return a * x + (x < c ? x : c);
}

NUNA_HD inline ItemRange items_of(const Place& pl, int64_t b, int64_t G) {
    ItemRange r;
    if (pl.mode == kPlaceLinear) {
        r.first = b;
        r.end = pl.start[kNumXcd];
        r.stride = G;
        return r;
    }
    const int64_t x = b & (kNumXcd - 1);
    const int64_t k = b >> 3;
    r.first = pl.start[x] + k;
    r.end = pl.start[x + 1];
    r.stride = (G - x + kNumXcd - 1) >> 3;
    return r;
}

// Host: placement table for `groups` groups of `group_size` items.
inline Place make_place_uniform(int mode, int64_t G, int64_t groups, int64_t group_size) {
    Place pl{};
    pl.mode = mode;
    for (int x = 0; x <= kNumXcd; ++x) pl.start[x] = group_size * ((groups * wgs_before_xcd(x, G)) / G);
    pl.start[kNumXcd] = groups * group_size;
    return pl;
}

// Host: placement table for variable-size groups; group_start holds ngroups+1
// item offsets (the last one is the item count).
inline Place make_place_groups(int mode, int64_t G, const int64_t* group_start, int64_t ngroups) {
    Place pl{};
    pl.mode = mode;
    const int64_t nitems = group_start[ngroups];
    for (int x = 0; x < kNumXcd; ++x) {
        const int64_t target = nitems * wgs_before_xcd(x, G) / G;
        int64_t lo = 0, hi = ngroups;  // first group whose start is >= target
        while (lo < hi) {
            const int64_t mid = (lo + hi) / 2;
            if (group_start[mid] < target) lo = mid + 1;
            else hi = mid;
        }
        pl.start[x] = group_start[lo];
    }
    pl.start[0] = 0;
    pl.start[kNumXcd] = nitems;
    return pl;
}

}  // namespace nuna
