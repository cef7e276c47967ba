// Host-side layout derivation and launch planning of libstepq (see
// stepq_plan.h).  Plain C++: built with the host compiler, so that it also
// runs under the CPU sanitizers.
#include "stepq_plan.h"

#include <algorithm>
#include <utility>

namespace stepq {

namespace {

size_t round128(size_t x) { return (x + 127) & ~static_cast<size_t>(127); }

stepq_status failed(std::string *err, stepq_status s, const char *msg)
{
    if (err) *err = msg;
    return s;
}

bool pivot_uniform(int code) { return code > kPivotUniformBase && code <= kPivotUniformBase + kNumUniformLayouts; }

bool compiled(int code) { return code >= 1 && code <= kF16HeadLayout; }

bool compact_generic(const HeadInfo &hi)
{
    return hi.layout == 0 && hi.groups <= static_cast<uint32_t>(kCompactGroups) && hi.n16 <= kCompactPivots;
}

bool rowmix_head(const HeadInfo &hi, int dk)
{
    return hi.layout == 0 && dk == 128 && hi.n2 == 0 && hi.n16 <= kCompactPivots && hi.g8 == hi.n8 &&
           hi.g4 == (hi.n4 + 1) / 2 && hi.g2 == 0;
}

int32_t packed_counts(const HeadInfo &hi) { return static_cast<int32_t>(hi.n16 | (hi.n8 << 8) | (hi.n4 << 16)); }

bool fail_check(std::string *err, const std::string &msg)
{
    if (err) *err = msg;
    return false;
}

}  // namespace

stepq_status derive_layout(const stepq_pool_desc *d, std::vector<HeadInfo> *heads, std::vector<uint8_t> *perm,
                           size_t *slot_bytes, std::string *err)
{
    if (!d) return failed(err, STEPQ_E_INVALID, "descriptor is NULL");
    if (d->n_slots < 1 || d->n_v_heads < 1 || d->n_qk_heads < 1)
        return failed(err, STEPQ_E_INVALID, "n_slots, n_v_heads and n_qk_heads must be >= 1");
    if (d->n_v_heads % d->n_qk_heads != 0)
        return failed(err, STEPQ_E_INVALID, "n_v_heads must be a multiple of n_qk_heads");
    if (d->d_k < 1 || d->d_k > kMaxDk) return failed(err, STEPQ_E_UNSUPPORTED, "d_k must be in 1..128");
    if (d->d_v != 64 && d->d_v != 128) return failed(err, STEPQ_E_UNSUPPORTED, "d_v must be 64 or 128");
    if (!d->row_bits) return failed(err, STEPQ_E_INVALID, "row_bits is NULL");
    if (d->levels != STEPQ_LEVELS_ABSMAX && d->levels != STEPQ_LEVELS_POW2)
        return failed(err, STEPQ_E_INVALID, "levels must be STEPQ_LEVELS_ABSMAX or STEPQ_LEVELS_POW2");
    const int Hv = d->n_v_heads, dk = d->d_k, dv = d->d_v;
    heads->assign(Hv, HeadInfo{});
    perm->assign(static_cast<size_t>(Hv) * dk, 0);
    size_t off = 0;
    for (int h = 0; h < Hv; ++h) {
        const uint8_t *b = d->row_bits + static_cast<size_t>(h) * dk;
        int n16 = 0, n8 = 0, n4 = 0, n2 = 0;
        for (int i = 0; i < dk; ++i) {
            if (b[i] == 16) ++n16;
            else if (b[i] == 8) ++n8;
            else if (b[i] == 4) ++n4;
            else if (b[i] == 2) ++n2;
            else return failed(err, STEPQ_E_INVALID, "row_bits entries must be 2, 4, 8 or 16");
        }
        const bool f16_head = n16 == dk && dk == 128 && dv == 128;   // a whole FP16 head
        if (n16 > kMaxPivots && !f16_head)
            return failed(err, STEPQ_E_UNSUPPORTED,
                          "at most 32 pivot (16) rows per head, or all rows of a 128x128 head");
        int p = 0;
        for (int width : {16, 8, 4, 2})
            for (int i = 0; i < dk; ++i)
                if (b[i] == width) (*perm)[static_cast<size_t>(h) * dk + p++] = static_cast<uint8_t>(i);
        HeadInfo &hi = (*heads)[h];
        hi.n16 = static_cast<uint16_t>(n16);
        hi.n8 = static_cast<uint16_t>(n8);
        hi.n4 = static_cast<uint16_t>(n4);
        hi.n2 = static_cast<uint16_t>(n2);
        hi.g8 = static_cast<uint16_t>(n8);
        hi.g4 = static_cast<uint16_t>((n4 + 1) / 2);
        hi.g2 = static_cast<uint16_t>((n2 + 3) / 4);
        hi.layout = 0;
        // At d = 128, integer rows that fit a uniform mix (first in table
        // order) are stored in it: exactly, or, when pivot rows take some of
        // the 128, with each width class padded by empty groups.
        if (dv == 128 && dk == 128 && !f16_head)
            for (int L = 0; L < kNumUniformLayouts; ++L) {
                const UniformLayout &u = kUniformLayouts[L];
                if (8 * u.m8 < n8 || 16 * u.m4 < n4 || 32 * u.m2 < n2) continue;
                hi.g8 = static_cast<uint16_t>(8 * u.m8);
                hi.g4 = static_cast<uint16_t>(8 * u.m4);
                hi.g2 = static_cast<uint16_t>(8 * u.m2);
                if (n16 == 0) hi.layout = L + 1;
                else if (n16 <= kCompactPivots) hi.layout = kPivotUniformBase + L + 1;
                break;
            }
        hi.groups = static_cast<uint32_t>(hi.g8 + hi.g4 + hi.g2);
        if (f16_head) hi.layout = kF16HeadLayout;
        const size_t creg = round128(static_cast<size_t>(hi.groups) * dv);
        const size_t preg = round128(static_cast<size_t>(n16) * 2u * dv);
        const size_t tb = round128(creg + preg + 4u * static_cast<size_t>(dk) + 4u * static_cast<size_t>(dv));
        hi.piv_off = static_cast<uint32_t>(creg);
        hi.r_off = static_cast<uint32_t>(creg + preg);
        hi.tile_bytes = static_cast<uint32_t>(tb);
        hi.tile_off = static_cast<uint32_t>(off);
        // the compiled bodies address codes (or FP16 values), r and c from these sizes
        if (hi.layout > 0 && static_cast<int>(hi.layout) <= kNumUniformLayouts) {
            const UniformLayout &u = kUniformLayouts[hi.layout - 1];
            const uint32_t m = static_cast<uint32_t>(u.m8 + u.m4 + u.m2);
            if (hi.r_off != 1024u * m || hi.tile_bytes != 1024u * (m + 1))
                return failed(err, STEPQ_E_INVALID, "internal: uniform head layout does not match its tile size");
        }
        if (static_cast<int>(hi.layout) > kPivotUniformBase) {
            const UniformLayout &u = kUniformLayouts[hi.layout - kPivotUniformBase - 1];
            const uint32_t m = static_cast<uint32_t>(u.m8 + u.m4 + u.m2);
            if (hi.piv_off != 1024u * m || hi.r_off != 1024u * m + 256u * n16 || hi.tile_bytes != hi.r_off + 1024u)
                return failed(err, STEPQ_E_INVALID,
                              "internal: padded pivot head layout does not match its tile size");
        }
        if (static_cast<int>(hi.layout) == kF16HeadLayout &&
            (hi.piv_off != 0 || hi.r_off != 128u * 256u || hi.tile_bytes != 128u * 256u + 1024u))
            return failed(err, STEPQ_E_INVALID, "internal: FP16 head layout does not match its tile size");
        off += tb;
        // tile offsets inside a slot record are 32-bit
        if (off > UINT32_MAX) return failed(err, STEPQ_E_UNSUPPORTED, "slot record over 4 GiB: too many heads");
    }
    *slot_bytes = off;
    return STEPQ_OK;
}

FastDiv fast_div(uint32_t d)
{
    uint32_t sh = 0;
    while ((1ull << sh) < d) ++sh;
    const uint64_t m = ((1ull << 32) * ((1ull << sh) - d)) / d + 1;
    return FastDiv{static_cast<uint32_t>(m), sh};
}

uint32_t fixed_tile_bytes(int layout)
{
    if (layout >= 1 && layout <= kNumUniformLayouts) {
        const UniformLayout &u = kUniformLayouts[layout - 1];
        return 1024u * static_cast<uint32_t>(u.m8 + u.m4 + u.m2 + 1);
    }
    if (layout == kF16HeadLayout) return 128u * 256u + 1024u;
    return 0;
}

void plan_launches(const std::vector<HeadInfo> &heads, int dk, int dv, LaunchPlan *plan)
{
    *plan = LaunchPlan{};
    plan->layout = static_cast<int>(heads[0].layout);
    for (const HeadInfo &hi : heads)
        if (static_cast<int>(hi.layout) != plan->layout) plan->layout = 0;
    // padded pivot heads differ in their row counts, which travel in the head list
    if (plan->layout > kPivotUniformBase) plan->layout = 0;
    if (plan->layout != 0 || dv != 128) return;

    // one class per layout present; larger classes are launched first
    std::vector<std::pair<int, int>> cls;   // (-count, layout)
    std::vector<int> codes;
    for (int L = 0; L <= kF16HeadLayout; ++L) codes.push_back(L);
    for (int L = 1; L <= kNumUniformLayouts; ++L) codes.push_back(kPivotUniformBase + L);
    for (int L : codes) {
        int n = 0;
        for (const HeadInfo &hi : heads) n += static_cast<int>(hi.layout) == L;
        if (n > 0) cls.emplace_back(-n, L);
    }
    std::sort(cls.begin(), cls.end());
    for (const auto &c : cls) {
        int code = c.second;
        if (code == 0) {
            // the generic heads take the row-mix body when every one of them
            // is a compact 8/4-bit head with few pivot rows, else the compact
            // generic body when all of them fit it
            bool fits = true, rowmix = true;
            for (const HeadInfo &hi : heads) {
                if (hi.layout != 0) continue;
                fits = fits && compact_generic(hi);
                rowmix = rowmix && rowmix_head(hi, dk);
            }
            if (rowmix) code = kRowMix;
            else if (fits) code = kCompactGeneric;
        }
        plan->cls_code.push_back(code);
        plan->cls_off.push_back(static_cast<int>(plan->order.size()));
        plan->cls_cnt.push_back(-c.first);
        for (size_t h = 0; h < heads.size(); ++h) {
            const HeadInfo &hi = heads[h];
            if (static_cast<int>(hi.layout) != c.second) continue;
            plan->order.push_back({static_cast<int32_t>(h), hi.tile_off, static_cast<int32_t>(hi.layout),
                                   packed_counts(hi)});
        }
    }
    // one uniform class of layout 1 or 2 whose other classes are its padded
    // pivot heads, compact generic or whole FP16 heads: a decode step is one
    // combined launch
    int L = 0, others = 0, pivots = 0;
    bool fits = true, f16 = false;
    for (int code : plan->cls_code)
        if (code == 1 || code == 2) {
            if (L != 0) fits = false;
            L = code;
        }
    for (int code : plan->cls_code) {
        if (code == 1 || code == 2) continue;
        if (code == kCompactGeneric || code == kF16HeadLayout || (L != 0 && code == kPivotUniformBase + L)) {
            ++others;
            f16 = f16 || code == kF16HeadLayout;
            pivots += code == kPivotUniformBase + L;
        } else {
            fits = false;
        }
    }
    // several classes that all have compiled bodies (uniform mixes, their
    // padded pivot heads, whole FP16 heads): one launch of those bodies only,
    // which fits fewer registers than the ones below.  The head list keeps
    // the classes together: tiles of one kind in runs stream better than
    // interleaved kinds.
    bool all_compiled = plan->cls_code.size() > 1, piv = false;
    for (int code : plan->cls_code) {
        all_compiled = all_compiled && (compiled(code) || pivot_uniform(code));
        piv = piv || pivot_uniform(code);
    }
    if (fits && L != 0 && others > 0 && others == pivots)
        plan->mixed_code = kMixedPivotBase + L;       // one uniform mix and its pivot heads: one body
    else if (all_compiled)
        plan->mixed_code = piv ? kMultiPivot : kMultiUniform;
    else if (fits && L != 0 && others > 0)
        plan->mixed_code = (f16 ? kMixedF16Base : kMixedBase) + L;
}

bool decode_body_runs(int code, const HeadInfo &hi, int dk)
{
    const int L = static_cast<int>(hi.layout);
    if (compiled(code) || pivot_uniform(code)) return L == code;
    if (code > kMixedPivotBase && code <= kMixedPivotBase + 2) {
        const int u = code - kMixedPivotBase;
        return L == u || L == kPivotUniformBase + u;
    }
    if (code > kMixedF16Base && code <= kMixedF16Base + 2) {
        const int u = code - kMixedF16Base;
        return L == u || L == kPivotUniformBase + u || L == kF16HeadLayout || compact_generic(hi);
    }
    if (code > kMixedBase && code <= kMixedBase + 2) {
        const int u = code - kMixedBase;
        return L == u || L == kPivotUniformBase + u || compact_generic(hi);
    }
    if (code == kMultiUniform) return compiled(L);
    if (code == kMultiPivot) return compiled(L) || pivot_uniform(L);
    if (code == kRowMix) return rowmix_head(hi, dk);
    if (code == kCompactGeneric) return compact_generic(hi);
    if (code == 0) return L == 0;
    return false;
}

bool refit_combined(int mixed_code)
{
    return mixed_code == kMultiUniform || (mixed_code > kMixedPivotBase && mixed_code <= kMixedPivotBase + 2);
}

bool refit_body_runs(int code, const HeadInfo &hi, int dk)
{
    const int L = static_cast<int>(hi.layout);
    if (compiled(code)) return L == code;    // whole FP16 heads take their decode body in every mode
    // the row-mix class has a refitting body of its own (the dual-axis fit;
    // the row-absmax step takes the generic body, which runs these heads too)
    if (code == kRowMix) return rowmix_head(hi, dk);
    // the combined launch of the uniform refitting bodies and whole FP16 heads
    if (code == kMultiUniform) return compiled(L);
    // padded pivot heads have a refitting body of their own (the dual-axis
    // fit; the row-absmax step takes the generic body, which runs them too),
    // which also runs the heads of their uniform layout in one launch
    if (pivot_uniform(code)) return L == code;
    if (code > kMixedPivotBase && code <= kMixedPivotBase + 2) {
        const int u = code - kMixedPivotBase;
        return L == u || L == kPivotUniformBase + u;
    }
    // every other code runs the generic refitting body, which reads the
    // head's own record (the tight layout, or a padded uniform mix)
    return !compiled(L);
}

bool check_plan(const LaunchPlan &plan, const std::vector<HeadInfo> &heads, int dk, int dv, size_t slot_bytes,
                std::string *err)
{
    const int Hv = static_cast<int>(heads.size());
    if (Hv < 1) return fail_check(err, "no heads");
    // the head records tile the slot record
    size_t off = 0;
    for (int h = 0; h < Hv; ++h) {
        const HeadInfo &hi = heads[h];
        const std::string at = "head " + std::to_string(h) + ": ";
        if (hi.tile_off != off) return fail_check(err, at + "tile offset is not the end of the previous tile");
        if (hi.tile_bytes == 0 || hi.tile_bytes % 128 != 0) return fail_check(err, at + "tile size not a multiple of 128");
        if (hi.groups != static_cast<uint32_t>(hi.g8 + hi.g4 + hi.g2)) return fail_check(err, at + "group count");
        if (hi.n16 + hi.n8 + hi.n4 + hi.n2 != dk) return fail_check(err, at + "row counts do not sum to d_k");
        if (hi.g8 < hi.n8 || 2 * hi.g4 < hi.n4 || 4 * hi.g2 < hi.n2)
            return fail_check(err, at + "row groups do not hold the head's rows");
        if (static_cast<uint64_t>(hi.groups) * dv > hi.piv_off)
            return fail_check(err, at + "codes region overlaps the pivot rows");
        if (hi.piv_off + 2ull * dv * hi.n16 > hi.r_off) return fail_check(err, at + "pivot rows overlap r");
        if (hi.r_off + 4ull * (dk + dv) > hi.tile_bytes) return fail_check(err, at + "r and c run past the tile");
        off += hi.tile_bytes;
    }
    if (off != slot_bytes) return fail_check(err, "the tiles do not fill the slot record");

    if (plan.order.empty()) {
        if (!plan.cls_code.empty() || plan.mixed_code != 0)
            return fail_check(err, "classes or a combined launch without a head list");
        const uint32_t tb = fixed_tile_bytes(plan.layout);
        for (int h = 0; h < Hv; ++h) {
            const HeadInfo &hi = heads[h];
            const std::string at = "head " + std::to_string(h) + ": ";
            if (static_cast<int>(hi.layout) != plan.layout)
                return fail_check(err, at + "layout differs from the single launch's");
            if (tb != 0 && (hi.tile_bytes != tb || hi.tile_off != static_cast<uint64_t>(tb) * h))
                return fail_check(err, at + "not where the body's fixed tile size puts it");
            if (!decode_body_runs(plan.layout, hi, dk) || !refit_body_runs(plan.layout, hi, dk))
                return fail_check(err, at + "the single launch's body does not run it");
        }
        if (plan.layout == 0 && dv == 128) return fail_check(err, "a generic pool at d_v = 128 needs a head list");
        return true;
    }

    if (plan.order.size() != static_cast<size_t>(Hv)) return fail_check(err, "head list does not hold every head");
    std::vector<char> seen(Hv, 0);
    for (size_t e = 0; e < plan.order.size(); ++e) {
        const LaunchHead &lh = plan.order[e];
        const std::string at = "head list entry " + std::to_string(e) + ": ";
        if (lh.h < 0 || lh.h >= Hv) return fail_check(err, at + "head index out of range");
        if (seen[lh.h]) return fail_check(err, at + "head listed twice");
        seen[lh.h] = 1;
        const HeadInfo &hi = heads[lh.h];
        if (lh.tile_off != hi.tile_off) return fail_check(err, at + "tile offset differs from the head record");
        if (static_cast<uint64_t>(lh.tile_off) + hi.tile_bytes > slot_bytes)
            return fail_check(err, at + "tile runs past the slot record");
        if (lh.layout != static_cast<int32_t>(hi.layout)) return fail_check(err, at + "layout differs");
        if (lh.counts != packed_counts(hi)) return fail_check(err, at + "row counts differ");
    }
    const size_t nc = plan.cls_code.size();
    if (nc == 0 || plan.cls_off.size() != nc || plan.cls_cnt.size() != nc)
        return fail_check(err, "class tables missing or of different lengths");
    int next = 0;
    for (size_t c = 0; c < nc; ++c) {
        const std::string at = "class " + std::to_string(c) + ": ";
        if (plan.cls_off[c] != next || plan.cls_cnt[c] < 1)
            return fail_check(err, at + "not the next non-empty slice of the head list");
        next += plan.cls_cnt[c];
        if (next > Hv) return fail_check(err, at + "runs past the head list");
        for (int e = plan.cls_off[c]; e < next; ++e) {
            const HeadInfo &hi = heads[plan.order[e].h];
            if (!decode_body_runs(plan.cls_code[c], hi, dk))
                return fail_check(err, at + "its decode body does not run head " + std::to_string(plan.order[e].h));
            if (!refit_body_runs(plan.cls_code[c], hi, dk))
                return fail_check(err, at + "its refitting body does not run head " + std::to_string(plan.order[e].h));
        }
    }
    if (next != Hv) return fail_check(err, "the classes do not cover the head list");
    if (plan.mixed_code != 0)
        for (const LaunchHead &lh : plan.order) {
            if (!decode_body_runs(plan.mixed_code, heads[lh.h], dk))
                return fail_check(err, "the combined launch's body does not run head " + std::to_string(lh.h));
            // the refit takes the combined launches that refit_combined names
            if (refit_combined(plan.mixed_code) && !refit_body_runs(plan.mixed_code, heads[lh.h], dk))
                return fail_check(err, "the combined refitting launch does not run head " + std::to_string(lh.h));
        }
    return true;
}

}  // namespace stepq
