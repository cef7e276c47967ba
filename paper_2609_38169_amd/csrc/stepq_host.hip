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
#include "stepq_plan.h"

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
    stepq::LaunchPlan plan;           // the decode launches of a step (stepq_plan.h)
    stepq::LaunchHead *d_head_order = nullptr;  // plan.order on the device
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

// Validate a descriptor and derive the layout tables (include/stepq.h).
stepq_status build_layout(const stepq_pool_desc *d, std::vector<HeadInfo> *heads, std::vector<uint8_t> *perm,
                          size_t *slot_bytes)
{
    std::string err;
    const stepq_status st = stepq::derive_layout(d, heads, perm, slot_bytes, &err);
    return st == STEPQ_OK ? st : fail(st, err);
}

using stepq::fast_div;

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

stepq_status stepq_pool_plan(const stepq_pool_desc *desc, uint32_t flags, stepq_launch_desc *launches,
                             int32_t max_launches, int32_t *n_launches, int32_t *head_order)
{
    if (!n_launches) return fail(STEPQ_E_INVALID, "n_launches is NULL");
    *n_launches = 0;
    if (max_launches < 0 || (max_launches > 0 && !launches)) return fail(STEPQ_E_INVALID, "bad launches buffer");
    if (flags & ~static_cast<uint32_t>(STEPQ_STEP_KDA_GATE | STEPQ_STEP_REFIT | STEPQ_STEP_ROW_ABSMAX |
                                       STEPQ_STEP_ADJACENT_SLOTS))
        return fail(STEPQ_E_INVALID, "unknown decode-step flags");
    std::vector<HeadInfo> heads;
    std::vector<uint8_t> perm;
    size_t sb = 0;
    stepq_status st = build_layout(desc, &heads, &perm, &sb);
    if (st != STEPQ_OK) return st;
    stepq::LaunchPlan plan;
    stepq::plan_launches(heads, desc->d_k, desc->d_v, &plan);
    std::string why;
    if (!stepq::check_plan(plan, heads, desc->d_k, desc->d_v, sb, &why))
        return fail(STEPQ_E_INVALID, "internal: launch plan check failed: " + why);
    const int Hv = desc->n_v_heads;
    std::vector<stepq_launch_desc> out;
    if (plan.mixed_code != 0 && !(flags & (STEPQ_STEP_REFIT | STEPQ_STEP_ROW_ABSMAX)))
        out.push_back({plan.mixed_code, 0, Hv});
    else if (plan.cls_code.empty())
        out.push_back({plan.layout, 0, Hv});
    else
        for (size_t c = 0; c < plan.cls_code.size(); ++c)
            out.push_back({plan.cls_code[c], plan.cls_off[c], plan.cls_cnt[c]});
    for (size_t i = 0; i < out.size() && static_cast<int32_t>(i) < max_launches; ++i) launches[i] = out[i];
    *n_launches = static_cast<int32_t>(out.size());
    if (head_order)
        for (int x = 0; x < Hv; ++x) head_order[x] = plan.order.empty() ? x : plan.order[x].h;
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
    // the decode launches, checked against the head records before any
    // allocation or launch: a plan that would send a workgroup outside its
    // tile, or a head to a body that does not run it, is refused here
    stepq::plan_launches(p->heads, p->dk, p->dv, &p->plan);
    std::string why;
    if (!stepq::check_plan(p->plan, p->heads, p->dk, p->dv, p->slot_bytes, &why)) {
        delete p;
        return fail(STEPQ_E_INVALID, "internal: launch plan check failed: " + why);
    }
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
    if (e == hipSuccess && !p->plan.order.empty()) {
        const auto &order = p->plan.order;
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

stepq_status stepq_pool_set_row_weight(stepq_pool *p, const float *row_weight, void *stream)
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
    stepq_status st = check_device(p);
    if (st != STEPQ_OK) return st;
    // in stream order: after the steps already enqueued on the stream, before
    // later ones; the host waits for this stream only (phys must outlive the copy)
    auto s = static_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(p->d_roww, phys.data(), sizeof(float) * phys.size(), hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
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
    const stepq::LaunchPlan &plan = p->plan;
    // the combined launches the refit has bodies for: several uniform layouts
    // and whole FP16 heads, or one uniform layout and its padded pivot heads
    const bool refit_multi = (flags & STEPQ_STEP_REFIT) && stepq::refit_combined(plan.mixed_code);
    if ((plan.mixed_code != 0 && !(flags & (STEPQ_STEP_REFIT | STEPQ_STEP_ROW_ABSMAX))) || refit_multi) {
        // uniform heads share one launch with compact generic and whole FP16
        // heads; with the refit, the heads of refit_combined's launches share
        // one launch of the refitting bodies
        a.head_list = p->d_head_order;
        a.n_heads = p->Hv;
        a.div_heads = fast_div(static_cast<uint32_t>(p->Hv));
        e = launch(plan.mixed_code);
    } else if (plan.cls_code.empty()) {
        a.head_list = nullptr;
        a.n_heads = p->Hv;
        a.div_heads = fast_div(static_cast<uint32_t>(p->Hv));
        e = launch(plan.layout);
    } else {
        // a mixed pool: one launch per layout class, each with its own register budget
        for (size_t c = 0; c < plan.cls_code.size() && e == hipSuccess; ++c) {
            a.head_list = p->d_head_order + plan.cls_off[c];
            a.n_heads = plan.cls_cnt[c];
            a.div_heads = fast_div(static_cast<uint32_t>(plan.cls_cnt[c]));
            e = launch(plan.cls_code[c]);
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

stepq_status stepq_decode_stream_ref(stepq_pool *p, const int32_t *slot_ids, int32_t batch, const void *q,
                                     const void *k, const void *v, const void *alpha, const void *beta,
                                     stepq_dtype act_dtype, uint32_t flags, float *o, void *stream)
{
    stepq_status st = common_checks(p, slot_ids, batch);
    if (st != STEPQ_OK) return st;
    if (act_dtype != STEPQ_F32 && act_dtype != STEPQ_BF16) return fail(STEPQ_E_INVALID, "unknown activation dtype");
    if (flags & ~static_cast<uint32_t>(STEPQ_STEP_ADJACENT_SLOTS))
        return fail(STEPQ_E_INVALID, "the memory-only reference takes STEPQ_STEP_ADJACENT_SLOTS only");
    if (batch == 0) return STEPQ_OK;
    if (!q || !k || !v || !alpha || !beta || !o) return fail(STEPQ_E_INVALID, "NULL activation or output pointer");
    auto s = static_cast<hipStream_t>(stream);
    st = check_slots(p, slot_ids, batch, s);
    if (st != STEPQ_OK) return st;
    stepq::DecodeArgs a{};
    a.pool = view(p);
    a.slot_ids = slot_ids;
    a.q = q;
    a.k = k;
    a.v = v;
    a.alpha = alpha;
    a.beta = beta;
    a.o = o;
    a.batch = batch;
    a.launch_order = (flags & STEPQ_STEP_ADJACENT_SLOTS) ? 1 : 0;
    // one launch over every head, in the order of the combined decode launch
    a.head_list = p->plan.order.empty() ? nullptr : p->d_head_order;
    a.n_heads = p->Hv;
    a.div_heads = fast_div(static_cast<uint32_t>(p->Hv));
    const hipError_t e = stepq::launch_stream_ref(a, act_dtype == STEPQ_BF16, s);
    return e == hipSuccess ? STEPQ_OK : hip_fail(e, "reference launch");
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
