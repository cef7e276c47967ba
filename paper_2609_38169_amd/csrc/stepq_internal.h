// Internal types shared by the host side and the kernels of libstepq.
// The pool layout they describe is defined in include/stepq.h.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime.h>

#include "stepq_layout.h"

namespace stepq {

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
// kPivotUniformBase + L; the refit takes its row-mix body for kRowMix and
// one launch over the uniform refitting bodies and the FP16-head body for
// kMultiUniform (the row-absmax step launches such pools per class).
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
// Memory-only reference of a decode launch: the same tiles, order and
// memory traffic (codes rewritten unchanged, o zeroed), no arithmetic.
hipError_t launch_stream_ref(const DecodeArgs &a, bool bf16, hipStream_t stream);
hipError_t launch_tile_op(const TileArgs &a, TileOp op, hipStream_t stream);

}  // namespace stepq
