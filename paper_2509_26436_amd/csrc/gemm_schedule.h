// Work schedule of the W4A4 GEMM (internal; compiled for host and device).
//
// The GEMM runs a persistent grid of `blocks` workgroups, each one walking a
// list of segments (a tile and a range of its 64-groups) as one continuous
// pipeline:
//   * tiles [0, sk_first) are whole-tile work: workgroup b takes tiles
//     b, b + blocks, b + 2 blocks, ... (the order a tile grid is dispatched in);
//   * the remaining tiles [sk_first, sk_first + sk_tiles) are cut along K:
//     their (tile, group) units, tile-major, are split into sk_blocks
//     contiguous ranges of q or q + 1 units, one per workgroup (stream-K), so
//     that every workgroup ends at nearly the same time whatever the number
//     of tiles.
// A range can begin and end inside a tile, so a tile of the split part may be
// shared by several workgroups: each one stores its partial fp32 sum in a
// slot of the caller's workspace and the last one to arrive adds them up (in
// a fixed order) and writes the output.  A workgroup has at most two partial
// segments (its first and its last), hence two slots.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define QUARTZ_HD __host__ __device__
#else
#define QUARTZ_HD
#endif

namespace quartz {

struct GemmSchedule {
    int32_t tiles_n;     // output tiles along N
    int32_t groups;      // K / 64
    int32_t blocks;      // persistent grid size
    int32_t sk_first;    // tiles below this are whole-tile work
    int32_t sk_tiles;    // tiles in the split part (0: nothing is split)
    int32_t sk_blocks;   // workgroups sharing the split part (<= blocks)
    int32_t sk_q;        // units per workgroup: sk_q + 1 for b < sk_r, sk_q otherwise
    int32_t sk_r;
};

struct GemmSegment {
    int32_t tile;        // linear tile index, row-major over (tile row, tile column)
    int32_t g0, g1;      // groups [g0, g1) of the tile
    int32_t sk_tile;     // index in the split part if the segment is partial, else -1
    int32_t slot;        // workspace slot of a partial segment, else -1
};

QUARTZ_HD inline int32_t sk_min(int32_t a, int32_t b) { return a < b ? a : b; }

// whole tiles of workgroup b
QUARTZ_HD inline int32_t dp_count(const GemmSchedule& s, int32_t b)
{
    return b < s.sk_first ? (s.sk_first - 1 - b) / s.blocks + 1 : 0;
}

// first unit of workgroup b's range in the split part (b may be >= sk_blocks)
QUARTZ_HD inline int32_t sk_start(const GemmSchedule& s, int32_t b)
{
    if (b >= s.sk_blocks)
        return s.sk_tiles * s.groups;
    return b * s.sk_q + sk_min(b, s.sk_r);
}

// workgroup whose range holds unit u (0 <= u < sk_tiles * groups)
QUARTZ_HD inline int32_t sk_block_of(const GemmSchedule& s, int32_t u)
{
    const int32_t big = s.sk_r * (s.sk_q + 1);
    return u < big ? u / (s.sk_q + 1) : s.sk_r + (u - big) / s.sk_q;
}

// segment j of workgroup b; false once the workgroup has no more
QUARTZ_HD inline bool gemm_segment(const GemmSchedule& s, int32_t b, int32_t j, GemmSegment& sg)
{
    const int32_t nd = dp_count(s, b);
    if (j < nd) {
        sg.tile = j * s.blocks + b;
        sg.g0 = 0;
        sg.g1 = s.groups;
        sg.sk_tile = -1;
        sg.slot = -1;
        return true;
    }
    const int32_t jj = j - nd;
    const int32_t u0 = sk_start(s, b), u1 = sk_start(s, b + 1);
    if (u0 >= u1)
        return false;
    const int32_t t = u0 / s.groups + jj;
    const int32_t tu = t * s.groups;
    if (tu >= u1)
        return false;
    sg.tile = s.sk_first + t;
    sg.g0 = jj == 0 ? u0 - tu : 0;
    sg.g1 = sk_min(s.groups, u1 - tu);
    const bool partial = sg.g0 > 0 || sg.g1 < s.groups;
    sg.sk_tile = partial ? t : -1;
    sg.slot = partial ? 2 * b + (jj > 0 ? 1 : 0) : -1;
    return true;
}

// Incremental walk over workgroup b's segments, as the kernel does it: the
// same sequence as gemm_segment(s, b, 0), gemm_segment(s, b, 1), ... with
// divisions only when it starts and where it enters the split part.
struct GemmCursor {
    GemmSegment sg;      // current segment
    int32_t j;           // its index
    int32_t tm, tn;      // tile row and column of sg.tile
    int32_t dp_left;     // whole tiles after this one (-1: in the split part)
    int32_t u1;          // end of the workgroup's split range (units)
    int32_t dm, dn;      // blocks / tiles_n, blocks % tiles_n
};

QUARTZ_HD inline bool cursor_split_begin(const GemmSchedule& s, int32_t b, GemmCursor& c)
{
    const int32_t u0 = sk_start(s, b);
    c.u1 = sk_start(s, b + 1);
    c.dp_left = -1;
    if (u0 >= c.u1)
        return false;
    const int32_t t = u0 / s.groups;
    c.sg.tile = s.sk_first + t;
    c.tm = c.sg.tile / s.tiles_n;
    c.tn = c.sg.tile - c.tm * s.tiles_n;
    c.sg.g0 = u0 - t * s.groups;
    c.sg.g1 = sk_min(s.groups, c.u1 - t * s.groups);
    const bool partial = c.sg.g0 > 0 || c.sg.g1 < s.groups;
    c.sg.sk_tile = partial ? t : -1;
    c.sg.slot = partial ? 2 * b : -1;
    return true;
}

QUARTZ_HD inline bool cursor_begin(const GemmSchedule& s, int32_t b, GemmCursor& c)
{
    c.j = 0;
    c.dm = s.blocks / s.tiles_n;
    c.dn = s.blocks - c.dm * s.tiles_n;
    const int32_t nd = dp_count(s, b);
    if (nd == 0)
        return cursor_split_begin(s, b, c);
    c.dp_left = nd - 1;
    c.sg.tile = b;
    c.tm = b / s.tiles_n;
    c.tn = b - c.tm * s.tiles_n;
    c.sg.g0 = 0;
    c.sg.g1 = s.groups;
    c.sg.sk_tile = -1;
    c.sg.slot = -1;
    return true;
}

QUARTZ_HD inline bool cursor_next(const GemmSchedule& s, int32_t b, GemmCursor& c)
{
    ++c.j;
    if (c.dp_left > 0) {
        --c.dp_left;
        c.sg.tile += s.blocks;
        c.tm += c.dm;
        c.tn += c.dn;
        if (c.tn >= s.tiles_n) {
            c.tn -= s.tiles_n;
            ++c.tm;
        }
        return true;
    }
    if (c.dp_left == 0)
        return cursor_split_begin(s, b, c);
    const int32_t t = c.sg.tile - s.sk_first + 1;          // next tile of the split part
    if (t * s.groups >= c.u1)
        return false;
    ++c.sg.tile;
    if (++c.tn == s.tiles_n) {
        c.tn = 0;
        ++c.tm;
    }
    c.sg.g0 = 0;
    c.sg.g1 = sk_min(s.groups, c.u1 - t * s.groups);
    const bool partial = c.sg.g1 < s.groups;
    c.sg.sk_tile = partial ? t : -1;
    c.sg.slot = partial ? 2 * b + 1 : -1;
    return true;
}

// The pipeline runs every segment in a whole number of 3-step rounds (the
// three LDS stages), the steps past its groups doing nothing, so that each
// segment's first group lands in stage 0.
constexpr int32_t kPipelineStages = 3;

QUARTZ_HD inline int32_t padded_steps(int32_t groups)
{
    return (groups + kPipelineStages - 1) / kPipelineStages * kPipelineStages;
}

// pipeline steps of workgroup b
QUARTZ_HD inline int32_t gemm_steps(const GemmSchedule& s, int32_t b)
{
    GemmCursor c;
    int32_t n = 0;
    for (bool ok = cursor_begin(s, b, c); ok; ok = cursor_next(s, b, c))
        n += padded_steps(c.sg.g1 - c.sg.g0);
    return n;
}

// workgroups [b_first, b_last] that share tile t of the split part
QUARTZ_HD inline void sk_contributors(const GemmSchedule& s, int32_t t, int32_t& b_first,
                                      int32_t& b_last)
{
    b_first = sk_block_of(s, t * s.groups);
    b_last = sk_block_of(s, t * s.groups + s.groups - 1);
}

// slot in which workgroup b keeps its partial sum of split tile t
QUARTZ_HD inline int32_t sk_slot(const GemmSchedule& s, int32_t b, int32_t t)
{
    return 2 * b + (t > sk_start(s, b) / s.groups ? 1 : 0);
}

}  // namespace quartz
