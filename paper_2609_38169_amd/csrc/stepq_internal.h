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
    uint32_t r_off;       // byte offset of r inside the tile (= padded codes region)
    uint16_t n8, n4, n2;  // rows of each width
    uint16_t g8, g4, g2;  // row groups of each width
    uint32_t groups;      // g8 + g4 + g2
};

// Row-constant table index space: 8-bit rows, then the two slots of every
// 4-bit group, then the four slots of every 2-bit group (empty slots
// included), so group g / slot s maps to one index without a lookup.
// Its size is at most d_k + 4.
constexpr int kMaxDk = 128;
constexpr int kSlotTable = kMaxDk + 4;

struct PoolView {
    uint8_t *base;
    uint64_t slot_bytes;
    const HeadInfo *heads;   // [Hv], device
    const uint8_t *perm;     // [Hv][d_k] physical row -> logical row, device
    int32_t n_slots, Hv, Hqk, dk, dv;
};

struct DecodeArgs {
    PoolView pool;
    const int32_t *slot_ids;
    const void *q, *k, *v, *alpha, *beta;
    float *o;
    int32_t batch;
};

enum class TileOp : int { Load = 0, Import = 1, Export = 2, Dequant = 3 };

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
};

hipError_t launch_decode(const DecodeArgs &a, bool bf16, hipStream_t stream);
hipError_t launch_tile_op(const TileArgs &a, TileOp op, hipStream_t stream);

}  // namespace stepq
