// Host-side layout derivation and launch planning of libstepq (plain C++, no
// HIP): the per-head layout records of a pool descriptor, the decode
// launches a pool issues per step, and a check that every launch's grid and
// head list stay inside what its kernel body reads.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "stepq.h"
#include "stepq_layout.h"

namespace stepq {

// The decode launches of a pool, fixed when the pool is created.
//  - order empty: one launch without a head list covers every head, in head
//    order; every head has layout `layout` (a compiled body's fixed tile size
//    then places head h at h * tile size), or d_v = 64 (generic body).
//  - order non-empty (d_v = 128 pools of several layouts): the heads grouped
//    by class, larger classes first.  Class c is order[cls_off[c] ..
//    cls_off[c] + cls_cnt[c]) and launches the body cls_code[c]; when
//    mixed_code is not 0, a frozen decode step is one launch of that body
//    over the whole of order instead (the refitting steps always launch per
//    class).
struct LaunchPlan {
    int layout = 0;
    std::vector<LaunchHead> order;
    std::vector<int> cls_code, cls_off, cls_cnt;
    int mixed_code = 0;
};

// Validate a descriptor and derive the per-head layout records and the
// physical -> logical row permutation ([Hv][d_k]) of the layout that
// include/stepq.h defines.  On failure *err names the reason.
stepq_status derive_layout(const stepq_pool_desc *d, std::vector<HeadInfo> *heads, std::vector<uint8_t> *perm,
                           size_t *slot_bytes, std::string *err);

// The launch plan of a pool with these head records.
void plan_launches(const std::vector<HeadInfo> &heads, int dk, int dv, LaunchPlan *plan);

// Whether the frozen-step decode body of launch code `code` handles head
// `hi`, and the same for the refitting bodies (refit and row-absmax).
bool decode_body_runs(int code, const HeadInfo &hi, int dk);
bool refit_body_runs(int code, const HeadInfo &hi, int dk);
// Whether the refit runs a plan's combined launch (mixed_code) as one
// launch of its refitting bodies (else it launches per class).
bool refit_combined(int mixed_code);

// Tile size that the compiled body of layout code L (1 .. kF16HeadLayout)
// assumes for every head when it runs without a head list; 0 otherwise.
uint32_t fixed_tile_bytes(int layout);

// Check a plan against the head records before anything is launched with it:
//  - the head records tile the slot record: consecutive tiles, each region
//    (codes, pivot rows, r, c) inside its tile, the last tile ending at
//    slot_bytes;
//  - without a head list, every head has the plan's layout and sits where
//    the body's fixed tile size puts it;
//  - with one, the list holds every head exactly once, each entry's head
//    index, tile offset, layout and row counts are those of its head record,
//    and tile offset + tile size <= slot_bytes;
//  - the classes cut the list into consecutive, non-empty slices that cover
//    it, and the body each launch takes (per class, frozen and refitting;
//    the combined launch over the whole list) handles every head it gets.
// Returns false with the first violation in *err.
bool check_plan(const LaunchPlan &plan, const std::vector<HeadInfo> &heads, int dk, int dv, size_t slot_bytes,
                std::string *err);

// Constants for n / d by multiply-high in the kernels (FastDiv, d >= 1);
// exact for 0 <= n < 2^31.
FastDiv fast_div(uint32_t d);

}  // namespace stepq
