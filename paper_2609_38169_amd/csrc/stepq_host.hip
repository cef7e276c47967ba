// Host side of libstepq: the C ABI declared in include/stepq.h.
// Argument checking, the per-head layout tables, launches.
#include <algorithm>
#include <cstdlib>
#include <cstdint>
#include <cstring>
#include <string>
#include <cmath>
#include <vector>

#include "stepq.h"
#include "stepq_internal.h"

using stepq::HeadInfo;

struct stepq_pool {
    int32_t n_slots, Hv, Hqk, dk, dv;
    std::vector<uint8_t> bits;        // [Hv][dk]
    std::vector<HeadInfo> heads;      // [Hv]
    std::vector<uint8_t> perm;        // [Hv][dk] physical -> logical
    size_t slot_bytes = 0, pool_bytes = 0;
    uint8_t *mem = nullptr;
    bool owns_mem = false;
    HeadInfo *d_heads = nullptr;
    uint8_t *d_perm = nullptr;
    float *d_roww = nullptr;          // [Hv][dk] row-impact factors, physical order
    int device = 0;
    int levels = STEPQ_LEVELS_ABSMAX; // level normalisation of the codes
    int layout = 0;                   // uniform layout of every head, or 0
    // Layout classes of a mixed pool at d_v = 128: heads grouped by their
    // uniform layout (1-5), or the generic heads (0, or kCompactGeneric when
    // all of them fit the compact body); one decode launch per class.  Empty
    // when one launch covers every head.
    std::vector<int> cls_layout, cls_off, cls_cnt;
    // kMixedBase + L when the classes are uniform layout L (1 or 2) plus
    // compact generic and/or whole FP16 heads: then a decode step (without
    // refit) is one launch over the whole head list.  0 otherwise.
    int mixed_code = 0;
    stepq::LaunchHead *d_head_order = nullptr;  // [Hv] heads ordered by class, device
};

namespace {

thread_local std::string g_err;

stepq_status fail(stepq_status s, const std::string &msg)
{
    g_err = msg;
    return s;
}

stepq_status hip_fail(hipError_t e, const char *what)
{
    return fail(STEPQ_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

size_t round128(size_t x) { return (x + 127) & ~static_cast<size_t>(127); }

// Validate a descriptor and derive the layout tables (include/stepq.h).
stepq_status build_layout(const stepq_pool_desc *d, std::vector<HeadInfo> *heads, std::vector<uint8_t> *perm,
                          size_t *slot_bytes)
{
    if (!d) return fail(STEPQ_E_INVALID, "descriptor is NULL");
    if (d->n_slots < 1 || d->n_v_heads < 1 || d->n_qk_heads < 1)
        return fail(STEPQ_E_INVALID, "n_slots, n_v_heads and n_qk_heads must be >= 1");
    if (d->n_v_heads % d->n_qk_heads != 0)
        return fail(STEPQ_E_INVALID, "n_v_heads must be a multiple of n_qk_heads");
    if (d->d_k < 1 || d->d_k > stepq::kMaxDk) return fail(STEPQ_E_UNSUPPORTED, "d_k must be in 1..128");
    if (d->d_v != 64 && d->d_v != 128) return fail(STEPQ_E_UNSUPPORTED, "d_v must be 64 or 128");
    if (!d->row_bits) return fail(STEPQ_E_INVALID, "row_bits is NULL");
    if (d->levels != STEPQ_LEVELS_ABSMAX && d->levels != STEPQ_LEVELS_POW2)
        return fail(STEPQ_E_INVALID, "levels must be STEPQ_LEVELS_ABSMAX or STEPQ_LEVELS_POW2");
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
            else return fail(STEPQ_E_INVALID, "row_bits entries must be 2, 4, 8 or 16");
        }
        const bool f16_head = n16 == dk && dk == 128 && dv == 128;   // a whole FP16 head
        if (n16 > stepq::kMaxPivots && !f16_head)
            return fail(STEPQ_E_UNSUPPORTED, "at most 32 pivot (16) rows per head, or all rows of a 128x128 head");
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
            for (int L = 0; L < stepq::kNumUniformLayouts; ++L) {
                const stepq::UniformLayout &u = stepq::kUniformLayouts[L];
                if (8 * u.m8 < n8 || 16 * u.m4 < n4 || 32 * u.m2 < n2) continue;
                hi.g8 = static_cast<uint16_t>(8 * u.m8);
                hi.g4 = static_cast<uint16_t>(8 * u.m4);
                hi.g2 = static_cast<uint16_t>(8 * u.m2);
                if (n16 == 0) hi.layout = L + 1;
                else if (n16 <= stepq::kCompactPivots) hi.layout = stepq::kPivotUniformBase + L + 1;
                break;
            }
        hi.groups = static_cast<uint32_t>(hi.g8 + hi.g4 + hi.g2);
        if (f16_head) hi.layout = stepq::kF16HeadLayout;
        const size_t creg = round128(static_cast<size_t>(hi.groups) * dv);
        const size_t preg = round128(static_cast<size_t>(n16) * 2u * dv);
        const size_t tb = round128(creg + preg + 4u * static_cast<size_t>(dk) + 4u * static_cast<size_t>(dv));
        hi.piv_off = static_cast<uint32_t>(creg);
        hi.r_off = static_cast<uint32_t>(creg + preg);
        hi.tile_bytes = static_cast<uint32_t>(tb);
        hi.tile_off = static_cast<uint32_t>(off);
        // the compiled bodies address codes (or FP16 values), r and c from these sizes
        if (hi.layout > 0 && static_cast<int>(hi.layout) <= stepq::kNumUniformLayouts) {
            const stepq::UniformLayout &u = stepq::kUniformLayouts[hi.layout - 1];
            const uint32_t m = static_cast<uint32_t>(u.m8 + u.m4 + u.m2);
            if (hi.r_off != 1024u * m || hi.tile_bytes != 1024u * (m + 1))
                return fail(STEPQ_E_INVALID, "internal: uniform head layout does not match its tile size");
        }
        if (static_cast<int>(hi.layout) > stepq::kPivotUniformBase) {
            const stepq::UniformLayout &u = stepq::kUniformLayouts[hi.layout - stepq::kPivotUniformBase - 1];
            const uint32_t m = static_cast<uint32_t>(u.m8 + u.m4 + u.m2);
            if (hi.piv_off != 1024u * m || hi.r_off != 1024u * m + 256u * n16 || hi.tile_bytes != hi.r_off + 1024u)
                return fail(STEPQ_E_INVALID, "internal: padded pivot head layout does not match its tile size");
        }
        if (static_cast<int>(hi.layout) == stepq::kF16HeadLayout &&
            (hi.piv_off != 0 || hi.r_off != 128u * 256u || hi.tile_bytes != 128u * 256u + 1024u))
            return fail(STEPQ_E_INVALID, "internal: FP16 head layout does not match its tile size");
        off += tb;
        // tile offsets inside a slot record are 32-bit
        if (off > UINT32_MAX) return fail(STEPQ_E_UNSUPPORTED, "slot record over 4 GiB: too many heads");
    }
    *slot_bytes = off;
    return STEPQ_OK;
}

stepq::FastDiv fast_div(uint32_t d)
{
    uint32_t sh = 0;
    while ((1ull << sh) < d) ++sh;
    const uint64_t m = ((1ull << 32) * ((1ull << sh) - d)) / d + 1;
    return stepq::FastDiv{static_cast<uint32_t>(m), sh};
}

stepq::PoolView view(const stepq_pool *p)
{
    stepq::PoolView v;
    v.base = p->mem;
    v.slot_bytes = p->slot_bytes;
    v.heads = p->d_heads;
    v.perm = p->d_perm;
    v.roww = p->d_roww;
    v.n_slots = p->n_slots;
    v.Hv = p->Hv;
    v.Hqk = p->Hqk;
    v.dk = p->dk;
    v.dv = p->dv;
    v.div_hv = fast_div(static_cast<uint32_t>(p->Hv));
    v.div_g = fast_div(static_cast<uint32_t>(p->Hv / p->Hqk));
    // per width 8 / 4 / 2: q = level * iq; nu = 1 / iq; fq = 2^(b-8) / iq
    const int widths[3] = {8, 4, 2};
    for (int w = 0; w < 3; ++w) {
        const int b = widths[w];
        const float qb = static_cast<float>((1 << (b - 1)) - 1);
        const float p2 = std::ldexp(1.0f, b - 8);       // 2^(b-8)
        if (p->levels == STEPQ_LEVELS_POW2) {
            v.lv.iq[w] = p2;
            v.lv.nu[w] = 1.0f / p2;
            v.lv.fq[w] = 1.0f;
        } else {
            v.lv.iq[w] = qb;
            v.lv.nu[w] = 1.0f / qb;
            v.lv.fq[w] = p2 / qb;
        }
    }
    return v;
}

bool debug_checks()
{
    const char *e = std::getenv("STEPQ_DEBUG");
    return e && e[0] == '1';
}

stepq_status check_device(const stepq_pool *p)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != p->device) return fail(STEPQ_E_INVALID, "the pool lives on another device than the current one");
    return STEPQ_OK;
}

// STEPQ_DEBUG=1: slot ids distinct and in range (synchronising host copy).
stepq_status check_slots(const stepq_pool *p, const int32_t *ids, int32_t n, hipStream_t s)
{
    if (!debug_checks() || n == 0) return STEPQ_OK;
    std::vector<int32_t> h(n);
    hipError_t e = hipStreamSynchronize(s);
    if (e == hipSuccess) e = hipMemcpy(h.data(), ids, sizeof(int32_t) * n, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "slot id check");
    std::vector<uint8_t> seen(p->n_slots, 0);
    for (int32_t i = 0; i < n; ++i) {
        if (h[i] < 0 || h[i] >= p->n_slots) return fail(STEPQ_E_INVALID, "slot id out of range");
        if (seen[h[i]]) return fail(STEPQ_E_INVALID, "slot id repeated within one call");
        seen[h[i]] = 1;
    }
    return STEPQ_OK;
}

// One launch covers n x Hv tiles of 256 work-items, and a dispatch counts its
// work-items in 32 bits.
constexpr int64_t kMaxTilesPerCall = int64_t(1) << 24;

stepq_status common_checks(const stepq_pool *p, const int32_t *ids, int32_t n)
{
    if (!p) return fail(STEPQ_E_INVALID, "pool is NULL");
    if (n < 0) return fail(STEPQ_E_INVALID, "negative count");
    if (n > p->n_slots) return fail(STEPQ_E_INVALID, "more slots requested than the pool holds");
    if (static_cast<int64_t>(n) * p->Hv > kMaxTilesPerCall)
        return fail(STEPQ_E_UNSUPPORTED, "more than 2^24 (slot, head) tiles in one call: split the batch");
    if (n > 0 && !ids) return fail(STEPQ_E_INVALID, "slot_ids is NULL");
    return check_device(p);
}

}  // namespace

extern "C" {

const char *stepq_last_error(void) { return g_err.c_str(); }

stepq_status stepq_pool_bytes(const stepq_pool_desc *desc, size_t *pool_bytes, size_t *slot_bytes)
{
    std::vector<HeadInfo> heads;
    std::vector<uint8_t> perm;
    size_t sb = 0;
    stepq_status st = build_layout(desc, &heads, &perm, &sb);
    if (st != STEPQ_OK) return st;
    if (pool_bytes) *pool_bytes = sb * static_cast<size_t>(desc->n_slots);
    if (slot_bytes) *slot_bytes = sb;
    return STEPQ_OK;
}

stepq_status stepq_pool_create(const stepq_pool_desc *desc, void *device_mem, size_t device_mem_bytes,
                               stepq_pool **out)
{
    if (!out) return fail(STEPQ_E_INVALID, "out is NULL");
    *out = nullptr;
    auto *p = new stepq_pool;
    stepq_status st = build_layout(desc, &p->heads, &p->perm, &p->slot_bytes);
    if (st != STEPQ_OK) {
        delete p;
        return st;
    }
    p->n_slots = desc->n_slots;
    p->levels = desc->levels;
    p->Hv = desc->n_v_heads;
    p->Hqk = desc->n_qk_heads;
    p->dk = desc->d_k;
    p->dv = desc->d_v;
    p->bits.assign(desc->row_bits, desc->row_bits + static_cast<size_t>(p->Hv) * p->dk);
    p->layout = static_cast<int>(p->heads[0].layout);
    for (const HeadInfo &hi : p->heads)
        if (static_cast<int>(hi.layout) != p->layout) p->layout = 0;
    // padded pivot heads differ in their row counts, which travel in the head list
    if (p->layout > stepq::kPivotUniformBase) p->layout = 0;
    p->pool_bytes = p->slot_bytes * static_cast<size_t>(p->n_slots);
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) {
        delete p;
        return hip_fail(e, "hipGetDevice");
    }
    if (device_mem) {
        if (reinterpret_cast<uintptr_t>(device_mem) % 256 != 0) {
            delete p;
            return fail(STEPQ_E_INVALID, "device_mem must be 256-byte aligned");
        }
        if (device_mem_bytes < p->pool_bytes) {
            delete p;
            return fail(STEPQ_E_INVALID, "device_mem is smaller than stepq_pool_bytes()");
        }
        p->mem = static_cast<uint8_t *>(device_mem);
    } else {
        e = hipMalloc(reinterpret_cast<void **>(&p->mem), p->pool_bytes);
        if (e != hipSuccess) {
            delete p;
            return fail(STEPQ_E_NOMEM, std::string("pool allocation: ") + hipGetErrorString(e));
        }
        p->owns_mem = true;
    }
    e = hipMalloc(reinterpret_cast<void **>(&p->d_heads), sizeof(HeadInfo) * p->heads.size());
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&p->d_perm), p->perm.size());
    if (e == hipSuccess)
        e = hipMemcpy(p->d_heads, p->heads.data(), sizeof(HeadInfo) * p->heads.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(p->d_perm, p->perm.data(), p->perm.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&p->d_roww), sizeof(float) * p->perm.size());
    if (e == hipSuccess) {
        const std::vector<float> ones(p->perm.size(), 1.0f);
        e = hipMemcpy(p->d_roww, ones.data(), sizeof(float) * ones.size(), hipMemcpyHostToDevice);
    }
    if (e == hipSuccess && p->layout == 0 && p->dv == 128) {
        // one class per layout present; larger classes are launched first
        std::vector<stepq::LaunchHead> order;
        std::vector<std::pair<int, int>> cls;   // (-count, layout)
        std::vector<int> codes;
        for (int L = 0; L <= stepq::kF16HeadLayout; ++L) codes.push_back(L);
        for (int L = 1; L <= stepq::kNumUniformLayouts; ++L) codes.push_back(stepq::kPivotUniformBase + L);
        for (int L : codes) {
            int n = 0;
            for (const HeadInfo &hi : p->heads) n += static_cast<int>(hi.layout) == L;
            if (n > 0) cls.emplace_back(-n, L);
        }
        std::sort(cls.begin(), cls.end());
        for (const auto &c : cls) {
            int code = c.second;
            if (code == 0) {
                // the generic heads take the row-mix body when every one of
                // them is a compact 8/4-bit head with few pivot rows, else the
                // compact generic body when all of them fit it
                bool fits = true, rowmix = p->dk == 128;
                for (const HeadInfo &hi : p->heads) {
                    if (hi.layout != 0) continue;
                    if (hi.groups > static_cast<uint32_t>(stepq::kCompactGroups) || hi.n16 > stepq::kCompactPivots)
                        fits = false;
                    if (hi.n2 != 0 || hi.n16 > stepq::kCompactPivots || hi.g8 != hi.n8 ||
                        hi.g4 != (hi.n4 + 1) / 2 || hi.g2 != 0)
                        rowmix = false;
                }
                if (rowmix) code = stepq::kRowMix;
                else if (fits) code = stepq::kCompactGeneric;
            }
            p->cls_layout.push_back(code);
            p->cls_off.push_back(static_cast<int>(order.size()));
            p->cls_cnt.push_back(-c.first);
            for (int h = 0; h < p->Hv; ++h) {
                const HeadInfo &hi = p->heads[h];
                if (static_cast<int>(hi.layout) != c.second) continue;
                const int32_t counts = static_cast<int32_t>(hi.n16 | (hi.n8 << 8) | (hi.n4 << 16));
                order.push_back({h, hi.tile_off, static_cast<int32_t>(hi.layout), counts});
            }
        }
        // one uniform class of layout 1 or 2 whose other classes are its
        // padded pivot heads, compact generic or whole FP16 heads: a decode
        // step is one combined launch
        int L = 0, others = 0, pivots = 0;
        bool fits = true, f16 = false;
        for (int code : p->cls_layout)
            if (code == 1 || code == 2) {
                if (L != 0) fits = false;
                L = code;
            }
        for (int code : p->cls_layout) {
            if (code == 1 || code == 2) continue;
            if (code == stepq::kCompactGeneric || code == stepq::kF16HeadLayout ||
                (L != 0 && code == stepq::kPivotUniformBase + L)) {
                ++others;
                f16 = f16 || code == stepq::kF16HeadLayout;
                pivots += code == stepq::kPivotUniformBase + L;
            } else {
                fits = false;
            }
        }
        // several classes that all have compiled bodies (uniform mixes,
        // their padded pivot heads, whole FP16 heads): one launch of those
        // bodies only, which fits fewer registers than the ones below.  The
        // head list keeps the classes together: tiles of one kind in runs
        // stream better than interleaved kinds.
        bool compiled = p->cls_layout.size() > 1, piv = false;
        for (int code : p->cls_layout) {
            const bool pc = code > stepq::kPivotUniformBase &&
                            code <= stepq::kPivotUniformBase + stepq::kNumUniformLayouts;
            compiled = compiled && ((code >= 1 && code <= stepq::kF16HeadLayout) || pc);
            piv = piv || pc;
        }
        if (fits && L != 0 && others > 0 && others == pivots)
            p->mixed_code = stepq::kMixedPivotBase + L;       // one uniform mix and its pivot heads: one body
        else if (compiled)
            p->mixed_code = piv ? stepq::kMultiPivot : stepq::kMultiUniform;
        else if (fits && L != 0 && others > 0)
            p->mixed_code = (f16 ? stepq::kMixedF16Base : stepq::kMixedBase) + L;
        e = hipMalloc(reinterpret_cast<void **>(&p->d_head_order), sizeof(stepq::LaunchHead) * order.size());
        if (e == hipSuccess)
            e = hipMemcpy(p->d_head_order, order.data(), sizeof(stepq::LaunchHead) * order.size(),
                          hipMemcpyHostToDevice);
    }
    if (e != hipSuccess) {
        stepq_pool_destroy(p);
        return fail(e == hipErrorOutOfMemory ? STEPQ_E_NOMEM : STEPQ_E_HIP,
                    std::string("layout tables: ") + hipGetErrorString(e));
    }
    *out = p;
    return STEPQ_OK;
}

void stepq_pool_destroy(stepq_pool *p)
{
    if (!p) return;
    (void)hipDeviceSynchronize();
    if (p->owns_mem && p->mem) (void)hipFree(p->mem);
    if (p->d_heads) (void)hipFree(p->d_heads);
    if (p->d_perm) (void)hipFree(p->d_perm);
    if (p->d_roww) (void)hipFree(p->d_roww);
    if (p->d_head_order) (void)hipFree(p->d_head_order);
    delete p;
}

void *stepq_pool_device_ptr(const stepq_pool *p) { return p ? p->mem : nullptr; }

stepq_status stepq_pool_set_row_weight(stepq_pool *p, const float *row_weight)
{
    if (!p || !row_weight) return fail(STEPQ_E_INVALID, "NULL pool or row_weight");
    std::vector<float> phys(p->perm.size());
    for (int h = 0; h < p->Hv; ++h)
        for (int x = 0; x < p->dk; ++x) {
            const size_t pi = static_cast<size_t>(h) * p->dk + x;
            const float wv = row_weight[static_cast<size_t>(h) * p->dk + p->perm[pi]];
            if (!(wv > 0.0f) || !std::isfinite(wv)) return fail(STEPQ_E_INVALID, "row weights must be finite and > 0");
            phys[pi] = wv;
        }
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != p->device) e = hipSetDevice(p->device);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpy(p->d_roww, phys.data(), sizeof(float) * phys.size(), hipMemcpyHostToDevice);
    if (cur != p->device) (void)hipSetDevice(cur);
    return e == hipSuccess ? STEPQ_OK : hip_fail(e, "row weight upload");
}

static stepq_status decode_step_impl(stepq_pool *p, const int32_t *slot_ids, int32_t batch, const void *q,
                                     const void *k, const void *v, const void *gate, const void *beta,
                                     stepq_dtype act_dtype, float *o, void *stream, uint32_t flags)
{
    stepq_status st = common_checks(p, slot_ids, batch);
    if (st != STEPQ_OK) return st;
    if (act_dtype != STEPQ_F32 && act_dtype != STEPQ_BF16) return fail(STEPQ_E_INVALID, "unknown activation dtype");
    if (flags & ~static_cast<uint32_t>(STEPQ_STEP_KDA_GATE | STEPQ_STEP_REFIT | STEPQ_STEP_ROW_ABSMAX |
                                       STEPQ_STEP_ADJACENT_SLOTS))
        return fail(STEPQ_E_INVALID, "unknown decode-step flags");
    if ((flags & STEPQ_STEP_REFIT) && (flags & STEPQ_STEP_ROW_ABSMAX))
        return fail(STEPQ_E_INVALID, "STEPQ_STEP_REFIT and STEPQ_STEP_ROW_ABSMAX exclude each other");
    if (batch == 0) return STEPQ_OK;
    if (!q || !k || !v || !gate || !beta || !o) return fail(STEPQ_E_INVALID, "NULL activation or output pointer");
    auto s = static_cast<hipStream_t>(stream);
    st = check_slots(p, slot_ids, batch, s);
    if (st != STEPQ_OK) return st;
    stepq::DecodeArgs a;
    a.pool = view(p);
    a.slot_ids = slot_ids;
    a.q = q;
    a.k = k;
    a.v = v;
    a.alpha = gate;
    a.beta = beta;
    a.o = o;
    a.batch = batch;
    const bool diag = (flags & STEPQ_STEP_KDA_GATE) != 0;
    const bool bf16 = act_dtype == STEPQ_BF16;
    a.f16_c_one = 0;
    a.launch_order = (flags & STEPQ_STEP_ADJACENT_SLOTS) ? 1 : 0;
    auto launch = [&](int layout) {
        if (layout == stepq::kF16HeadLayout) {
            // whole FP16 heads: no integer rows to fit, so every mode is the same update
            a.f16_c_one = (flags & STEPQ_STEP_ROW_ABSMAX) ? 1 : 0;
            const hipError_t r = stepq::launch_decode(a, bf16, diag, layout, s);
            a.f16_c_one = 0;
            return r;
        }
        return (flags & STEPQ_STEP_REFIT)        ? stepq::launch_decode_refit(a, bf16, diag, layout, s)
               : (flags & STEPQ_STEP_ROW_ABSMAX) ? stepq::launch_decode_rowmax(a, bf16, diag, layout, s)
                                                 : stepq::launch_decode(a, bf16, diag, layout, s);
    };
    hipError_t e = hipSuccess;
    if (p->mixed_code != 0 && !(flags & (STEPQ_STEP_REFIT | STEPQ_STEP_ROW_ABSMAX))) {
        // uniform heads share one launch with compact generic and whole FP16 heads
        a.head_list = p->d_head_order;
        a.n_heads = p->Hv;
        a.div_heads = fast_div(static_cast<uint32_t>(p->Hv));
        e = launch(p->mixed_code);
    } else if (p->cls_layout.empty()) {
        a.head_list = nullptr;
        a.n_heads = p->Hv;
        a.div_heads = fast_div(static_cast<uint32_t>(p->Hv));
        e = launch(p->layout);
    } else {
        // a mixed pool: one launch per layout class, each with its own register budget
        for (size_t c = 0; c < p->cls_layout.size() && e == hipSuccess; ++c) {
            a.head_list = p->d_head_order + p->cls_off[c];
            a.n_heads = p->cls_cnt[c];
            a.div_heads = fast_div(static_cast<uint32_t>(p->cls_cnt[c]));
            e = launch(p->cls_layout[c]);
        }
    }
    return e == hipSuccess ? STEPQ_OK : hip_fail(e, "decode launch");
}

stepq_status stepq_decode_step_ex(stepq_pool *p, const int32_t *slot_ids, int32_t batch, const void *q,
                                  const void *k, const void *v, const void *gate, const void *beta,
                                  stepq_dtype act_dtype, uint32_t flags, float *o, void *stream)
{
    return decode_step_impl(p, slot_ids, batch, q, k, v, gate, beta, act_dtype, o, stream, flags);
}

stepq_status stepq_decode_step(stepq_pool *p, const int32_t *slot_ids, int32_t batch, const void *q, const void *k,
                               const void *v, const void *alpha, const void *beta, stepq_dtype act_dtype, float *o,
                               void *stream)
{
    return decode_step_impl(p, slot_ids, batch, q, k, v, alpha, beta, act_dtype, o, stream, 0u);
}

stepq_status stepq_decode_step_kda(stepq_pool *p, const int32_t *slot_ids, int32_t batch, const void *q,
                                   const void *k, const void *v, const void *gate, const void *beta,
                                   stepq_dtype act_dtype, float *o, void *stream)
{
    return decode_step_impl(p, slot_ids, batch, q, k, v, gate, beta, act_dtype, o, stream, STEPQ_STEP_KDA_GATE);
}

static stepq_status tile_op(const stepq_pool *p, const int32_t *ids, int32_t n, stepq::TileArgs &a,
                            stepq::TileOp op, void *stream)
{
    auto s = static_cast<hipStream_t>(stream);
    stepq_status st = check_slots(p, ids, n, s);
    if (st != STEPQ_OK) return st;
    a.pool = view(p);
    a.slot_ids = ids;
    a.n = n;
    hipError_t e = stepq::launch_tile_op(a, op, s);
    return e == hipSuccess ? STEPQ_OK : hip_fail(e, "tile kernel launch");
}

stepq_status stepq_pool_load(stepq_pool *p, const int32_t *slot_ids, int32_t n, const float *state, const float *r,
                             const float *c, void *stream)
{
    stepq_status st = common_checks(p, slot_ids, n);
    if (st != STEPQ_OK) return st;
    if (n == 0) return STEPQ_OK;
    if (!state || !r || !c) return fail(STEPQ_E_INVALID, "NULL state or scale pointer");
    stepq::TileArgs a{};
    a.state = state;
    a.r_in = r;
    a.c_in = c;
    return tile_op(p, slot_ids, n, a, stepq::TileOp::Load, stream);
}

stepq_status stepq_pool_import(stepq_pool *p, const int32_t *slot_ids, int32_t n, const int8_t *codes,
                               const float *r, const float *c, void *stream)
{
    stepq_status st = common_checks(p, slot_ids, n);
    if (st != STEPQ_OK) return st;
    if (n == 0) return STEPQ_OK;
    if (!codes || !r || !c) return fail(STEPQ_E_INVALID, "NULL codes or scale pointer");
    stepq::TileArgs a{};
    a.codes_in = codes;
    a.r_in = r;
    a.c_in = c;
    return tile_op(p, slot_ids, n, a, stepq::TileOp::Import, stream);
}

stepq_status stepq_pool_export(const stepq_pool *p, const int32_t *slot_ids, int32_t n, int8_t *codes, float *r,
                               float *c, void *stream)
{
    stepq_status st = common_checks(p, slot_ids, n);
    if (st != STEPQ_OK) return st;
    if (n == 0) return STEPQ_OK;
    if (!codes || !r || !c) return fail(STEPQ_E_INVALID, "NULL output pointer");
    stepq::TileArgs a{};
    a.codes_out = codes;
    a.r_out = r;
    a.c_out = c;
    return tile_op(p, slot_ids, n, a, stepq::TileOp::Export, stream);
}

stepq_status stepq_pool_export_pivots(const stepq_pool *p, const int32_t *slot_ids, int32_t n, uint16_t *pivots,
                                      void *stream)
{
    stepq_status st = common_checks(p, slot_ids, n);
    if (st != STEPQ_OK) return st;
    if (n == 0) return STEPQ_OK;
    if (!pivots) return fail(STEPQ_E_INVALID, "NULL output pointer");
    stepq::TileArgs a{};
    a.piv_out = pivots;
    return tile_op(p, slot_ids, n, a, stepq::TileOp::ExportPivots, stream);
}

stepq_status stepq_pool_import_pivots(stepq_pool *p, const int32_t *slot_ids, int32_t n, const uint16_t *pivots,
                                      void *stream)
{
    stepq_status st = common_checks(p, slot_ids, n);
    if (st != STEPQ_OK) return st;
    if (n == 0) return STEPQ_OK;
    if (!pivots) return fail(STEPQ_E_INVALID, "NULL pivot pointer");
    stepq::TileArgs a{};
    a.piv_in = pivots;
    return tile_op(p, slot_ids, n, a, stepq::TileOp::ImportPivots, stream);
}

stepq_status stepq_pool_dequant(const stepq_pool *p, const int32_t *slot_ids, int32_t n, float *out, void *stream)
{
    stepq_status st = common_checks(p, slot_ids, n);
    if (st != STEPQ_OK) return st;
    if (n == 0) return STEPQ_OK;
    if (!out) return fail(STEPQ_E_INVALID, "NULL output pointer");
    stepq::TileArgs a{};
    a.deq_out = out;
    return tile_op(p, slot_ids, n, a, stepq::TileOp::Dequant, stream);
}

}  // extern "C"
