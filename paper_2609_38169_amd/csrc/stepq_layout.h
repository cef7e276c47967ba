// Layout types of libstepq shared by the host planning code and the
// kernels: per-head layout records, the uniform row-width mixes with
// compiled decode bodies, the launch codes, and the head list of a launch.
// Plain C++ (no HIP), so the planning code also builds with the host
// compiler alone.  The pool layout they describe is defined in
// include/stepq.h.
#pragma once

#include <stdint.h>

namespace stepq {


// Per value head: where its tile sits in a slot record and how its key rows
// are grouped by width.  Identical for every slot.
struct HeadInfo {
    uint32_t tile_off;    // byte offset of the tile inside a slot record
    uint32_t tile_bytes;  // record size (multiple of 128)
    uint32_t piv_off;     // byte offset of the pivot rows (= padded codes region)
    uint32_t r_off;       // byte offset of r inside the tile (after the pivot rows)
    uint16_t n16;         // pivot rows (binary16 values, physical rows 0 .. n16-1)
    uint16_t n8, n4, n2;  // integer rows of each width
    uint16_t g8, g4, g2;  // row groups of each width
    uint32_t groups;      // g8 + g4 + g2
    uint32_t layout;      // index into kUniformLayouts + 1, or 0 for the generic path
};

// Row-group mixes with a compile-time decode body at d_v = 128, in units of
// 8 row groups (one word-step of a 256-thread workgroup): {8-bit, 4-bit,
// 2-bit}.  Heads whose mix is listed keep their codes in registers between
// the two passes; any other mix takes the generic body.
struct UniformLayout {
    int m8, m4, m2;
};
constexpr UniformLayout kUniformLayouts[] = {
    {8, 4, 0},    // 64 rows @8 + 64 rows @4 (6 bits/element)
    {4, 2, 2},    // 32 @8 + 32 @4 + 64 @2 (4 bits/element)
    {16, 0, 0},   // all rows @8
    {0, 8, 0},    // all rows @4
    {0, 0, 4},    // all rows @2
};
constexpr int kNumUniformLayouts = sizeof(kUniformLayouts) / sizeof(kUniformLayouts[0]);
// Layout code of a head whose every row is an FP16 pivot (d_k = d_v = 128):
// its tile is the pivot region (32 KiB of binary16 values) and the unused r
// and c slots.
constexpr int kF16HeadLayout = kNumUniformLayouts + 1;

// Row-constant table index space: the slots of the 8-bit groups, then the
// two slots of every 4-bit group, then the four slots of every 2-bit group
// (empty slots included), so group g / slot s maps to one index without a
// lookup.  Its size is at most d_k + 4.
constexpr int kMaxDk = 128;
constexpr int kSlotTable = kMaxDk + 4;
constexpr int kMaxPivots = 32;    // FP16 pivot rows per head
// The compact generic decode body (layout code -1, d_v = 128) holds at most
// this many row groups and pivot rows per head, and fits 8 waves per SIMD.
constexpr int kCompactGeneric = -1;
// Layout code kMixedBase + L (L = 1, 2): heads of uniform layout L and
// compact generic heads in one decode launch; kMixedF16Base + L: the same
// with whole FP16 heads too (one more body, a few more registers).
constexpr int kMixedBase = 8;
constexpr int kMixedF16Base = 16;
constexpr int kCompactGroups = 96;
constexpr int kCompactPivots = 8;
// Layout code kPivotUniformBase + L: a head with 1 .. kCompactPivots FP16
// pivot rows whose integer rows are stored in uniform layout L, each width
// class padded with empty groups (zero codes) to L's group counts; the
// uniform decode body runs it with the pivot rows added, taking the row
// counts from its LaunchHead.
constexpr int kPivotUniformBase = 32;
// Layout code kMixedPivotBase + L (L = 1, 2): uniform layout-L heads and
// layout-L padded pivot heads only, in one decode launch of one body (a
// layout-L head is a padded pivot head without pivot rows).
constexpr int kMixedPivotBase = 24;
// Layout code kMultiUniform: heads of several compiled layouts (uniform
// mixes and whole FP16 heads) in one decode launch, each tile taking its
// own body; kMultiPivot: the same with padded pivot heads too (their body
// needs a few more registers).
constexpr int kMultiUniform = 40;
constexpr int kMultiPivot = 41;
// Layout code kRowMix: generic heads at d_k = d_v = 128 whose integer rows
// are 8- and 4-bit only, in any split, with at most kCompactPivots pivot
// rows, in the compact layout (row groups g8 = n8, g4 = ceil(n4 / 2)); one
// decode body runs them with the matrix cores whatever the split.  The
// heads keep layout 0 in their HeadInfo.
constexpr int kRowMix = 42;

// One value head of a decode launch over part of a pool's heads: its index
// and the byte offset of its tile within a slot record.
struct LaunchHead {
    int32_t h;
    uint32_t tile_off;
    int32_t layout;          // the head's uniform layout (1-based), or 0
    int32_t counts;          // n16 | n8 << 8 | n4 << 16 (read for padded pivot and uniform heads)
};

// n / d for 0 <= n < 2^31 by multiply-high (Granlund-Montgomery), with the
// constants prepared on the host so that uniform quotients stay scalar.
struct FastDiv {
    uint32_t mul, shift;
};

}  // namespace stepq
