// Internal types shared by the host side and the kernels of libstepq.
// The pool layout they describe is defined in include/stepq.h.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime.h>

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

// n / d for 0 <= n < 2^31 by multiply-high (Granlund-Montgomery), with the
// constants prepared on the host so that uniform quotients stay scalar.
struct FastDiv {
    uint32_t mul, shift;
};

// Per-width constants of the pool's level normalisation, index 0 / 1 / 2 for
// 8- / 4- / 2-bit rows.  The stored integer q of a row stands for the level
// z = q / iq (iq = q_b under N1, 2^(b-8) under N2, the paper's KDA
// codebook); nu = 1 / iq; fq = 2^(b-8) / iq turns an unpacked field
// 2^(8-b) q into z.
struct LevelTable {
    float iq[3], nu[3], fq[3];
};

struct PoolView {
    uint8_t *base;
    uint64_t slot_bytes;
    const HeadInfo *heads;   // [Hv], device
    const uint8_t *perm;     // [Hv][d_k] physical row -> logical row, device
    const float *roww;       // [Hv][d_k] row-impact factors w in physical row order, device
    int32_t n_slots, Hv, Hqk, dk, dv;
    FastDiv div_hv;          // divide by Hv
    FastDiv div_g;           // divide by Hv / Hqk
    LevelTable lv;
};

// One value head of a decode launch over part of a pool's heads: its index
// and the byte offset of its tile within a slot record.
struct LaunchHead {
    int32_t h;
    uint32_t tile_off;
    int32_t layout;          // the head's uniform layout (1-based), or 0
    int32_t counts;          // n16 | n8 << 8 | n4 << 16 (read for padded pivot and uniform heads)
};

struct DecodeArgs {
    PoolView pool;
    const int32_t *slot_ids;
    const void *q, *k, *v, *alpha, *beta;
    float *o;
    int32_t batch;
    // The value heads one launch covers: head_list[0 .. n_heads) (device),
    // or every head 0 .. Hv-1 in order when head_list is NULL (then every
    // head has the same tile size).  The grid is batch x n_heads workgroups.
    const LaunchHead *head_list;
    int32_t n_heads;
    FastDiv div_heads;       // divide by n_heads
    // Whole FP16 heads in a row-absmax step: their column factors become 1
    // (the baseline's c' = 1); their values update as in every other mode.
    int32_t f16_c_one;
    int32_t launch_order;    // 1: tile l of the launch is workgroup l (adjacent slots); 0: XCD runs
};

enum class TileOp : int { Load = 0, Import = 1, Export = 2, Dequant = 3, ExportPivots = 4, ImportPivots = 5 };

struct TileArgs {
    PoolView pool;
    const int32_t *slot_ids;
    int32_t n;
    const float *state;      // Load: [n][Hv][dk][dv]
    const int8_t *codes_in;  // Import
    const float *r_in;       // Load/Import: [n][Hv][dk] logical order
    const float *c_in;       // Load/Import: [n][Hv][dv]
    int8_t *codes_out;       // Export
    float *r_out, *c_out;    // Export
    float *deq_out;          // Dequant: [n][Hv][dk][dv]
    const uint16_t *piv_in;  // ImportPivots: [n][Hv][dk][dv] binary16, pivot rows read
    uint16_t *piv_out;       // ExportPivots: [n][Hv][dk][dv] binary16, pivot rows written, others 0
};

// pool_layout: the uniform layout (1-based) shared by every head of the
// launch (a.head_list), 0 for the generic body (irregular row-width mixes,
// FP16 pivot rows, d_v = 64), kCompactGeneric when every head of the launch
// fits the compact generic body's bounds, kF16HeadLayout for whole FP16
// heads, kPivotUniformBase + L for uniform-layout heads with pivot rows, or
// kMixedBase + L / kMixedF16Base + L (decode step only) for uniform layout-L
// heads mixed with such pivot heads, compact generic (and whole FP16) heads.
// The refitting steps take their generic body for kCompactGeneric and
// kPivotUniformBase + L.
// diag: a.alpha holds the channel-wise gate [batch][Hv][d_k] instead of the
// scalar gate [batch][Hv].
hipError_t launch_decode(const DecodeArgs &a, bool bf16, bool diag, int pool_layout, hipStream_t stream);
// The decode step followed by the online dual-axis refit of both scale
// vectors (the codes are requantized against the refitted scales, which
// replace the stored ones).
hipError_t launch_decode_refit(const DecodeArgs &a, bool bf16, bool diag, int pool_layout, hipStream_t stream);
// The decode step with the single-axis baseline's requantization: row
// factors r'_i = max_j |X_ij|, column factors 1.
hipError_t launch_decode_rowmax(const DecodeArgs &a, bool bf16, bool diag, int pool_layout, hipStream_t stream);
hipError_t launch_tile_op(const TileArgs &a, TileOp op, hipStream_t stream);

}  // namespace stepq
