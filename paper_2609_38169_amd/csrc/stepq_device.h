// Device-side building blocks of the decode kernels of libstepq (gfx950,
// wave64): activation loads, the XCD-aware tile order, row-group geometry,
// field unpacking, DPP wave reductions, the per-tile row constants and the
// column phase (S^T k, S^T q, residual, readout) shared by the frozen-scale
// and the refitting decode bodies.  Included by one or more kernel sources;
// everything here is internal to the including translation unit.
#pragma once

#include "stepq_internal.h"

namespace stepq {
namespace {

template <bool BF16>
__device__ __forceinline__ float act_ld(const void *p, size_t i)
{
    if constexpr (BF16) {
        const uint32_t u = static_cast<const uint16_t *>(p)[i];
        return __uint_as_float(u << 16);
    } else {
        return static_cast<const float *>(p)[i];
    }
}

// The code words of one tile, addressed through a buffer resource: the tile
// base is uniform (scalar registers) and each thread adds a 32-bit offset, so
// no 64-bit per-lane addresses are formed or kept live.  Word accesses stream
// past the caches: loads non-temporal, stores non-temporal at device scope
// (sc1 nt), the fastest policy measured for the in-place update on gfx950.
// Accesses beyond `bytes` read 0 and write nothing.
struct CodeWords {
    static constexpr int kLoad = 2;         // nt
    static constexpr int kStore = 16 | 2;   // sc1 nt
    __amdgpu_buffer_rsrc_t r;
    __device__ __forceinline__ CodeWords(const void *base, uint32_t bytes)
        : r(__builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, static_cast<int>(bytes), 0x00020000))
    {
    }
    __device__ __forceinline__ uint32_t load(int word) const
    {
        return __builtin_amdgcn_raw_buffer_load_b32(r, 4 * word, 0, kLoad);
    }
    __device__ __forceinline__ void store(int word, uint32_t v) const
    {
        __builtin_amdgcn_raw_buffer_store_b32(v, r, 4 * word, 0, kStore);
    }
    // Word tid + 256 m with the per-m part of the byte offset in the
    // instruction's immediate (m mod 4) and scalar (m / 4) offsets, so one
    // address register serves every m.  All such words lie inside the
    // record (the uniform bodies' tiles hold 256 words per m).
    __device__ __forceinline__ uint32_t load_m(int tid, int m) const
    {
        return __builtin_amdgcn_raw_buffer_load_b32(r, 4 * tid + 1024 * (m & 3), 4096 * (m >> 2), kLoad);
    }
    __device__ __forceinline__ void store_m(int tid, int m, uint32_t v) const
    {
        __builtin_amdgcn_raw_buffer_store_b32(v, r, 4 * tid + 1024 * (m & 3), 4096 * (m >> 2), kStore);
    }
};

// Workgroups are dispatched round-robin over the 8 XCDs.  Give each XCD a
// contiguous run of tiles so that value heads sharing a q/k head, and
// neighbouring slot records, are served from the same L2.
__device__ __forceinline__ int xcd_tile(int wg, int n)
{
    if ((n & 7) != 0) return wg;
    return (wg & 7) * (n >> 3) + (wg >> 3);
}

struct GroupRows {
    int bits;   // width of the group's rows
    int nslot;  // rows per group (8 / bits)
    int p0;     // physical row of slot 0
    int pend;   // one past the last physical row of this width
    int x0;     // row-table index of slot 0
};

// Physical rows: the n16 pivot rows first, then the integer rows 8, 4, 2;
// the row table and the groups cover the integer rows only.  A width class
// may hold more groups than its rows fill (g8 > n8, or a padded 4- or 2-bit
// class): its slots past the class's last row are empty (p0 + s >= pend)
// and their codes stay 0.
__device__ __forceinline__ GroupRows group_rows(const HeadInfo &hi, int g)
{
    const int P = hi.n16;
    if (g < hi.g8) return {8, 1, P + g, P + hi.n8, g};
    if (g < hi.g8 + hi.g4) {
        const int k = g - hi.g8;
        return {4, 2, P + hi.n8 + 2 * k, P + hi.n8 + hi.n4, hi.g8 + 2 * k};
    }
    const int k = g - hi.g8 - hi.g4;
    return {2, 4, P + hi.n8 + hi.n4 + 4 * k, P + hi.n8 + hi.n4 + hi.n2, hi.g8 + 2 * hi.g4 + 4 * k};
}

// Row-table slot x -> physical row (or -1 for an empty slot) and its width.
__device__ __forceinline__ int slot_row(const HeadInfo &hi, int x, int &bw)
{
    const int P = hi.n16;
    if (x < hi.g8) {
        bw = 8;
        return x < hi.n8 ? P + x : -1;
    }
    if (x < hi.g8 + 2 * hi.g4) {
        bw = 4;
        const int kk = x - hi.g8;
        return kk < hi.n4 ? P + hi.n8 + kk : -1;
    }
    bw = 2;
    if (x < hi.g8 + 2 * hi.g4 + 4 * hi.g2) {
        const int kk = x - hi.g8 - 2 * hi.g4;
        return kk < hi.n2 ? P + hi.n8 + hi.n4 + kk : -1;
    }
    return -1;
}

// The 4 fields of slot s of a word, each moved to the top of its byte
// (bytes of other slots cleared): a signed byte read then gives 2^(8-B) q.
template <int B>
__device__ __forceinline__ uint32_t slot_top(uint32_t w, int s)
{
    constexpr uint32_t top = ((0xFFu << (8 - B)) & 0xFFu) * 0x01010101u;
    return (w << (8 - B - s * B)) & top;
}

__device__ __forceinline__ float sbyte(uint32_t w, int e)
{
    return static_cast<float>(static_cast<int8_t>(static_cast<uint8_t>(w >> (8 * e))));
}

// A value every lane of the wavefront holds, moved to a scalar register.
__device__ __forceinline__ float uniform_f(float x)
{
    return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}

__device__ __forceinline__ int fdiv(int n, FastDiv d)
{
    const uint32_t u = static_cast<uint32_t>(n);
    return static_cast<int>((__umulhi(u, d.mul) + u) >> d.shift);
}

template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_term(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROWS, 0xF, false));
}

template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_bits(uint32_t x)
{
    return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), CTRL, ROWS, 0xF, false));
}

// Largest value over the 64 lanes of a wavefront, for x >= 0 (lanes a DPP
// step leaves out contribute 0); uniform result.  Non-negative floats order
// as their bit patterns do, so the steps are integer maxima.
__device__ __forceinline__ float wave_max(float x)
{
    uint32_t u = __float_as_uint(x);
    u = max(u, dpp_bits<0xB1, 0xF>(u));
    u = max(u, dpp_bits<0x4E, 0xF>(u));
    u = max(u, dpp_bits<0x141, 0xF>(u));
    u = max(u, dpp_bits<0x140, 0xF>(u));
    u = max(u, dpp_bits<0x142, 0xA>(u));
    u = max(u, dpp_bits<0x143, 0xC>(u));
    return __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(u), 63)));
}

// Sum over the 64 lanes of a wavefront with DPP row operations; the result
// is returned uniform (read from the last lane).
__device__ __forceinline__ float wave_sum(float x)
{
    x += dpp_term<0xB1, 0xF>(x);    // quad_perm [1,0,3,2]
    x += dpp_term<0x4E, 0xF>(x);    // quad_perm [2,3,0,1]: quad sums
    x += dpp_term<0x141, 0xF>(x);   // row_half_mirror: 8-lane sums
    x += dpp_term<0x140, 0xF>(x);   // row_mirror: 16-lane row sums
    x += dpp_term<0x142, 0xA>(x);   // row_bcast:15 into rows 1, 3
    x += dpp_term<0x143, 0xC>(x);   // row_bcast:31 into rows 2, 3
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

// ---------------------------------------------------------------------------
// decode step

template <int DV>
struct DecodeShared {
    float2 kq[kSlotTable];               // (k_i r_i f_i / q_b, q_i r_i f_i / q_b) per row-table slot
    float av[kSlotTable];                // beta k_i q_b / r_i
    float sk[kMaxDk], sq[kMaxDk];        // k, q of the tile in logical row order
    float sr[kMaxDk];                    // r in physical row order
    float sd[kMaxDk];                    // channel-wise gate d in logical row order (diagonal gate only)
    float al[kSlotTable];                // d_i 2^(b-8) per row-table slot (diagonal gate only)
    int sperm[kMaxDk];                   // logical row of each physical row
    float4 red[2][256 / (DV / 4)][DV / 4];
    float bcol[DV];                      // delta_j / c_j
    float kap[4];
    // FP16 pivot rows (generic bodies only), by physical row p < n16:
    // (k_i d_i, q_i d_i, d_i, beta k_i) with d_i the row's gate (alpha for GDN)
    float4 pvc[kMaxPivots];
    float cpiv[DV];                      // c_j, for the pivot rows' share of S^T k and S^T q
    // Uniform bodies: the row weights as binary16 A operands of the 4x4x4
    // matrix-core blocks, [slice][row group][type][row in group], types
    // 0/1 = k weight hi/lo, 2/3 = q weight hi/lo (prescaled by powers of two).
    // Row-mix body: [slice][word group][slot][type][word in group].
    union {
        alignas(16) _Float16 aop[8][4][4][4];
        alignas(16) _Float16 aopv[8][4][2][4][4];
    };
    float2 wmx[4];                       // per wavefront: largest |k weight|, |q weight|
};

struct TileCtx {
    int tile, b, h, hq;
    uint32_t off;            // byte offset of the tile in its slot record (uniform bodies)
    int layout;              // the head's uniform layout (1-based) or 0, when the launch has a head list
    int counts;              // n16 | n8 << 8 | n4 << 16 of the head (from the head list)
    HeadInfo hi;
    uint32_t *codes;
    const float *rr, *cc;
    float alpha, beta;
};

// The (request, value head) tile of this workgroup among the batch x
// n_heads tiles of the launch, in launch order or in XCD runs
// (a.launch_order); t.tile = b Hv + h indexes the activations.
// tile_bytes: the tile size shared by every head when the launch covers the
// whole pool in head order (a.head_list NULL).
__device__ __forceinline__ void tile_of(const DecodeArgs &a, uint32_t tile_bytes, TileCtx &t)
{
    const int l = a.launch_order ? static_cast<int>(blockIdx.x) : xcd_tile(blockIdx.x, a.batch * a.n_heads);
    t.b = fdiv(l, a.div_heads);
    int j = l - t.b * a.n_heads;
    if (a.head_list) {
        // rotate each request's heads by its index: tiles of one head then do
        // not recur at the same launch position modulo the CUs of an XCD
        j += t.b - a.n_heads * fdiv(j + t.b, a.div_heads);
        const LaunchHead lh = a.head_list[j];
        t.h = lh.h;
        t.off = lh.tile_off;
        t.layout = lh.layout;
        t.counts = lh.counts;
    } else {
        t.h = j;
        t.off = static_cast<uint32_t>(j) * tile_bytes;
        t.layout = 0;
        t.counts = 0;
    }
    t.tile = t.b * a.pool.Hv + t.h;
    t.hq = fdiv(t.h, a.pool.div_g);
}

// Per-tile operands of thread tid, loaded together at the start of a tile:
// k_i, q_i for logical row i = tid; r_p and the logical index of physical
// row p = tid; c_j, v_j for column j = tid.
struct RowColOps {
    float k, q, r, c, v;
    float d;                    // channel-wise gate of logical row tid (diagonal gate only)
    int perm;
};

template <bool BF16, bool DIAG, int DV>
__device__ __forceinline__ RowColOps load_ops(const DecodeArgs &a, int tile, int b, int hq, int h, const float *rr,
                                              const float *cc)
{
    const PoolView &P = a.pool;
    const int tid = threadIdx.x;
    RowColOps op{0.f, 0.f, 0.f, 0.f, 0.f, 1.f, 0};
    if (tid < P.dk) {
        if constexpr (DIAG) op.d = act_ld<BF16>(a.alpha, static_cast<size_t>(tile) * P.dk + tid);
        const size_t off = (static_cast<size_t>(b) * P.Hqk + hq) * P.dk + tid;
        op.k = act_ld<BF16>(a.k, off);
        op.q = act_ld<BF16>(a.q, off);
        op.r = rr[tid];
        op.perm = P.perm[h * P.dk + tid];
    }
    if (tid < DV) {
        op.c = cc[tid];
        op.v = act_ld<BF16>(a.v, static_cast<size_t>(tile) * DV + tid);
    }
    return op;
}

// Row constants into LDS, indexed by row-table slot, and q.k.  Two barriers;
// returns q.k.  Rows are read through the physical -> logical permutation
// from the LDS copy of k and q.
// SCALED: av and al come divided by the row width's clamp_scale, the form
// the frozen-scale requantization works in (requant_word).
template <bool DIAG, int DV, bool SCALED = false>
__device__ __forceinline__ float row_constants(const HeadInfo &hi, int dk, float alpha, float beta,
                                               const RowColOps &op, DecodeShared<DV> &sh, const LevelTable &lv)
{
    const int tid = threadIdx.x;
    if (tid < dk) {
        sh.sk[tid] = op.k;
        sh.sq[tid] = op.q;
        sh.sr[tid] = op.r;
        sh.sperm[tid] = op.perm;
        if constexpr (DIAG) sh.sd[tid] = op.d;
    }
    if (tid < DV) sh.cpiv[tid] = op.c;
    __syncthreads();
    float kq = 0.f;
    if (tid < hi.n16) {
        // pivot row p = tid (physical rows 0 .. n16-1); it also takes its share of q.k
        const int i = sh.sperm[tid];
        const float d = DIAG ? sh.sd[i] : alpha;
        const float kd = DIAG ? sh.sk[i] * d : sh.sk[i];     // the scalar gate is applied with the columns
        const float qd = DIAG ? sh.sq[i] * d : sh.sq[i];
        sh.pvc[tid] = make_float4(kd, qd, d, beta * sh.sk[i]);
        kq = sh.sq[i] * sh.sk[i];
    }
    if (tid < kSlotTable) {
        const int x = tid;
        int bw;
        const int p = slot_row(hi, x, bw);
        float kt = 0.f, qt = 0.f, av = 0.f, al = 0.f;
        if (p >= 0) {
            // slot x holds physical row p, whose r and permutation entry were
            // loaded by thread p
            const int i = sh.sperm[p];
            const float ki = sh.sk[i];
            const float qi = sh.sq[i];
            const float rp = sh.sr[p];
            // level of an unpacked field 2^(8-b) q: times fq (N1: 1/127, 1/112, 1/64)
            const int wi = bw == 8 ? 0 : (bw == 4 ? 1 : 2);
            const float qb = lv.iq[wi];
            const float fq = lv.fq[wi];
            const float di = DIAG ? sh.sd[i] : 1.0f;       // the gate folds into both row weights
            const float rs = rp * fq * di;
            kt = ki * rs;
            qt = qi * rs;
            const float sc = SCALED ? (bw == 8 ? 1.0f / 256.0f : (bw == 4 ? (1.0f / 14.0f) : 0.5f)) : 1.0f;
            av = beta * ki * (qb * sc) * __builtin_amdgcn_rcpf(rp);
            al = di * (bw == 8 ? sc : (bw == 4 ? (1.0f / 16.0f) * sc : (1.0f / 64.0f) * sc));
            kq += qi * ki;
        }
        sh.kq[x] = make_float2(kt, qt);
        sh.av[x] = av;
        if constexpr (DIAG) sh.al[x] = al;
    }
    kq = wave_sum(kq);
    if ((tid & 63) == 0) sh.kap[tid >> 6] = kq;
    __syncthreads();
    return (sh.kap[0] + sh.kap[1]) + (sh.kap[2] + sh.kap[3]);
}

// ---- FP16 pivot rows (generic bodies): thread (slice, cg) holds columns
// 4 cg .. 4 cg + 3 of pivot rows p = slice + NSL m, as 4 binary16 values.

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// PMAX: the most pivot rows a head of the launch may hold.
template <int DV, int PMAX = kMaxPivots>
struct PivotRegs {
    static constexpr int NSL = 256 / (DV / 4);
    static constexpr int M = (PMAX + NSL - 1) / NSL;
    u32x2 v[M];
};

template <int DV>
__device__ __forceinline__ u32x2 *pivot_ptr(const TileCtx &t, int p, int cg)
{
    return reinterpret_cast<u32x2 *>(reinterpret_cast<uint8_t *>(t.codes) + t.hi.piv_off +
                                     static_cast<uint32_t>(p) * (2u * DV) + 8u * static_cast<uint32_t>(cg));
}

template <int DV, int PMAX>
__device__ __forceinline__ void pivot_load(const TileCtx &t, int slice, int cg, PivotRegs<DV, PMAX> &pr)
{
#pragma unroll
    for (int m = 0; m < PivotRegs<DV, PMAX>::M; ++m) {
        const int p = slice + PivotRegs<DV, PMAX>::NSL * m;
        pr.v[m] = p < t.hi.n16 ? __builtin_nontemporal_load(pivot_ptr<DV>(t, p, cg)) : u32x2{0u, 0u};
    }
}

__device__ __forceinline__ float half_lo(uint32_t u) { return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(u))); }
__device__ __forceinline__ float half_hi(uint32_t u) { return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(u >> 16))); }

__device__ __forceinline__ uint32_t pack_halves(float a, float b)
{
    const uint16_t lo = __builtin_bit_cast(uint16_t, static_cast<_Float16>(a));   // round to nearest even
    const uint16_t hi = __builtin_bit_cast(uint16_t, static_cast<_Float16>(b));
    return static_cast<uint32_t>(lo) | (static_cast<uint32_t>(hi) << 16);
}

// The pivot rows' share of the column partials, pre-divided by c_j (the
// column phase multiplies the partials by c_j).
template <int DV, int PMAX>
__device__ __forceinline__ void pivot_acc(const TileCtx &t, int slice, int cg, const PivotRegs<DV, PMAX> &pr,
                                          const DecodeShared<DV> &sh, float (&acK)[4], float (&acQ)[4])
{
    if (t.hi.n16 == 0) return;
    const float4 c4 = *reinterpret_cast<const float4 *>(&sh.cpiv[4 * cg]);
    const float rc[4] = {__builtin_amdgcn_rcpf(c4.x), __builtin_amdgcn_rcpf(c4.y), __builtin_amdgcn_rcpf(c4.z),
                         __builtin_amdgcn_rcpf(c4.w)};
#pragma unroll
    for (int m = 0; m < PivotRegs<DV, PMAX>::M; ++m) {
        const int p = slice + PivotRegs<DV, PMAX>::NSL * m;
        if (p < t.hi.n16) {
            const float4 k = sh.pvc[p];
            const float sv[4] = {half_lo(pr.v[m].x), half_hi(pr.v[m].x), half_lo(pr.v[m].y), half_hi(pr.v[m].y)};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float s = sv[e] * rc[e];
                acK[e] = fmaf(k.x, s, acK[e]);
                acQ[e] = fmaf(k.y, s, acQ[e]);
            }
        }
    }
}

// New pivot values X_pj = d_i S_pj + beta k_i delta_j in binary16, stored in
// place (delta_j = bc_j c_j).
template <int DV, int PMAX>
__device__ __forceinline__ void pivot_update(const TileCtx &t, int slice, int cg, const PivotRegs<DV, PMAX> &pr,
                                             const DecodeShared<DV> &sh, const float (&bc)[4])
{
    if (t.hi.n16 == 0) return;
    const float4 c4 = *reinterpret_cast<const float4 *>(&sh.cpiv[4 * cg]);
    const float dl[4] = {bc[0] * c4.x, bc[1] * c4.y, bc[2] * c4.z, bc[3] * c4.w};
#pragma unroll
    for (int m = 0; m < PivotRegs<DV, PMAX>::M; ++m) {
        const int p = slice + PivotRegs<DV, PMAX>::NSL * m;
        if (p < t.hi.n16) {
            const float4 k = sh.pvc[p];
            const float sv[4] = {half_lo(pr.v[m].x), half_hi(pr.v[m].x), half_lo(pr.v[m].y), half_hi(pr.v[m].y)};
            float x[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = fmaf(k.w, dl[e], k.z * sv[e]);
            __builtin_nontemporal_store(u32x2{pack_halves(x[0], x[1]), pack_halves(x[2], x[3])},
                                        pivot_ptr<DV>(t, p, cg));
        }
    }
}

// A compact or padded pivot head's pivot row p = slice (at most one per
// thread: kCompactPivots = 8 slices): its share k_i S_pj / c_j and
// q_i S_pj / c_j of the column partials (the column phase multiplies by
// c_j), added to this thread's own in sh.red.
__device__ __forceinline__ void pivot_partials_slice(const TileCtx &t, int slice, int cg,
                                                     const PivotRegs<128, kCompactPivots> &pr, DecodeShared<128> &sh)
{
    static_assert(PivotRegs<128, kCompactPivots>::M == 1, "one pivot row per thread");
    if (slice < t.hi.n16) {
        const float4 c4 = *reinterpret_cast<const float4 *>(&sh.cpiv[4 * cg]);
        const uint32_t lo = pr.v[0].x, hi = pr.v[0].y;
        const float sv[4] = {half_lo(lo) * __builtin_amdgcn_rcpf(c4.x), half_hi(lo) * __builtin_amdgcn_rcpf(c4.y),
                             half_lo(hi) * __builtin_amdgcn_rcpf(c4.z), half_hi(hi) * __builtin_amdgcn_rcpf(c4.w)};
        const float4 kp = sh.pvc[slice];
        float4 &rk = sh.red[0][slice][cg];
        rk = make_float4(fmaf(kp.x, sv[0], rk.x), fmaf(kp.x, sv[1], rk.y), fmaf(kp.x, sv[2], rk.z),
                         fmaf(kp.x, sv[3], rk.w));
        float4 &rq = sh.red[1][slice][cg];
        rq = make_float4(fmaf(kp.y, sv[0], rq.x), fmaf(kp.y, sv[1], rq.y), fmaf(kp.y, sv[2], rq.z),
                         fmaf(kp.y, sv[3], rq.w));
    }
}

// A padded pivot head of uniform layout L (the tile of head list entry t):
// its row counts come from the head list (t.counts); its record holds the
// codes (1024 bytes per word-step), the n16 pivot rows (256 bytes each),
// then r and c.
template <int L>
__device__ __forceinline__ void padded_pivot_tile(const DecodeArgs &a, TileCtx &t, int slot)
{
    constexpr UniformLayout u = kUniformLayouts[L - 1];
    constexpr uint32_t piv_off = 1024u * (u.m8 + u.m4 + u.m2);
    const int n16 = t.counts & 0xff, n8 = (t.counts >> 8) & 0xff, n4 = (t.counts >> 16) & 0xff;
    t.hi.n16 = static_cast<uint16_t>(n16);
    t.hi.n8 = static_cast<uint16_t>(n8);
    t.hi.n4 = static_cast<uint16_t>(n4);
    t.hi.n2 = static_cast<uint16_t>(128 - n16 - n8 - n4);
    t.hi.g8 = static_cast<uint16_t>(8 * u.m8);
    t.hi.g4 = static_cast<uint16_t>(8 * u.m4);
    t.hi.g2 = static_cast<uint16_t>(8 * u.m2);
    t.hi.piv_off = piv_off;
    uint8_t *rec = a.pool.base + static_cast<uint64_t>(slot) * a.pool.slot_bytes + t.off;
    t.codes = reinterpret_cast<uint32_t *>(rec);
    t.rr = reinterpret_cast<const float *>(rec + piv_off + 256u * static_cast<uint32_t>(n16));
    t.cc = t.rr + 128;
}

// Power-of-two exponent that brings the largest weight m into [2^14, 2^15),
// where binary16 keeps its full precision and the hi/lo split below is
// exact to 22 significant bits.
__device__ __forceinline__ int weight_scale_exp(float m)
{
    const int e = __builtin_amdgcn_frexp_expf(m);   // m = f 2^e, f in [0.5, 1); 0 for m = 0
    return min(max(15 - e, -126), 126);
}

// Uniform layouts with the two matrix-vector products on the matrix cores.
// Row table slot = physical row = tid, as in row_constants_uniform; the k
// and q weights of each row are split into binary16 hi + lo parts (after
// the tile's prescales 2^ek, 2^eq) and written as the A operands of the
// 4x4x4 blocks of the thread's slice: aop[slice][group][type][row in
// group], the thread's 16 rows being its 8-bit rows, then the two slots of
// each 4-bit word, then the four slots of each 2-bit word (4 to a group).
// Two barriers; the operand table is complete only after one more.
// SCALED: av and al come divided by the row width's clamp_scale, the form
// the frozen-scale requantization works in (requant_field_p).
template <bool DIAG, int M8, int M4, int M2, int DV, bool SCALED = false>
__device__ __forceinline__ float row_constants_mfma(float beta, const RowColOps &op, DecodeShared<DV> &sh,
                                                    const LevelTable &lv, int &ek, int &eq)
{
    constexpr int X4 = 8 * M8, X2 = 8 * M8 + 16 * M4;
    const int tid = threadIdx.x;
    if (tid < 128) {
        sh.sk[tid] = op.k;
        sh.sq[tid] = op.q;
        if constexpr (DIAG) sh.sd[tid] = op.d;
    }
    __syncthreads();
    float kq = 0.f, kt = 0.f, qt = 0.f;
    if (tid < 128) {
        const int p = tid;
        const int wi = p < X4 ? 0 : (p < X2 ? 1 : 2);
        const float qb = lv.iq[wi];
        const float fq = lv.fq[wi];
        const float ki = sh.sk[op.perm];
        const float qi = sh.sq[op.perm];
        const float di = DIAG ? sh.sd[op.perm] : 1.0f;
        const float rs = op.r * fq * di;
        kt = ki * rs;
        qt = qi * rs;
        const float sc = SCALED ? (p < X4 ? 1.0f / 256.0f : (p < X2 ? (1.0f / 14.0f) : 0.5f)) : 1.0f;
        sh.av[p] = beta * ki * (qb * sc) * __builtin_amdgcn_rcpf(op.r);
        if constexpr (DIAG)
            sh.al[p] = di * (p < X4 ? sc : (p < X2 ? (1.0f / 16.0f) * sc : (1.0f / 64.0f) * sc));
        kq = qi * ki;
        // the rows live in wavefronts 0 and 1 only: the others skip the reductions
        kq = wave_sum(kq);
        const float mk = wave_max(fabsf(kt)), mq = wave_max(fabsf(qt));
        if ((tid & 63) == 0) {
            sh.kap[tid >> 6] = kq;
            sh.wmx[tid >> 6] = make_float2(mk, mq);
        }
    }
    __syncthreads();
    const float2 w0 = sh.wmx[0], w1 = sh.wmx[1];
    ek = __builtin_amdgcn_readfirstlane(weight_scale_exp(fmaxf(w0.x, w1.x)));
    eq = __builtin_amdgcn_readfirstlane(weight_scale_exp(fmaxf(w0.y, w1.y)));
    const float kappa = sh.kap[0] + sh.kap[1];
    if (tid < 128) {
        const int p = tid;
        int slice, ridx;
        if (p < X4) {
            slice = p & 7;
            ridx = p >> 3;
        } else if (p < X2) {
            const int c = (p - X4) >> 1;
            slice = c & 7;
            ridx = M8 + 2 * (c >> 3) + ((p - X4) & 1);
        } else {
            const int c = (p - X2) >> 2;
            slice = c & 7;
            ridx = M8 + 2 * M4 + 4 * (c >> 3) + ((p - X2) & 3);
        }
        const float ks = __builtin_amdgcn_ldexpf(kt, ek), qs = __builtin_amdgcn_ldexpf(qt, eq);
        const _Float16 kh = static_cast<_Float16>(ks), qh = static_cast<_Float16>(qs);
        const _Float16 kl = static_cast<_Float16>(ks - static_cast<float>(kh));
        const _Float16 ql = static_cast<_Float16>(qs - static_cast<float>(qh));
        _Float16(&dst)[4][4] = sh.aop[slice][ridx >> 2];
        dst[0][ridx & 3] = kh;
        dst[1][ridx & 3] = kl;
        dst[2][ridx & 3] = qh;
        dst[3][ridx & 3] = ql;
    }
    return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(kappa)));
}

// row_constants_mfma for a padded pivot head (layout code
// kPivotUniformBase + L): physical rows are the hi.n16 pivot rows, then the
// integer rows; table slot x = tid maps to its physical row through
// slot_row (empty slots get zero weights and update factors, so their zero
// codes stay zero).  Also the pivot rows' constants (pvc) and c (cpiv), as
// in row_constants.  Two barriers; the operand table needs one more.
template <bool DIAG, int M8, int M4, int M2, int DV, bool SCALED = false>
__device__ __forceinline__ float row_constants_mfma_piv(const HeadInfo &hi, float alpha, float beta,
                                                        const RowColOps &op, DecodeShared<DV> &sh,
                                                        const LevelTable &lv, int &ek, int &eq)
{
    const int tid = threadIdx.x;
    if (tid < 128) {
        sh.sk[tid] = op.k;
        sh.sq[tid] = op.q;
        sh.sr[tid] = op.r;
        sh.sperm[tid] = op.perm;
        sh.cpiv[tid] = op.c;
        if constexpr (DIAG) sh.sd[tid] = op.d;
    }
    __syncthreads();
    float kq = 0.f, kt = 0.f, qt = 0.f;
    if (tid < hi.n16) {
        // pivot row p = tid: its constants and its share of q.k
        const int i = sh.sperm[tid];
        const float d = DIAG ? sh.sd[i] : alpha;
        const float kd = DIAG ? sh.sk[i] * d : sh.sk[i];     // the scalar gate is applied with the columns
        const float qd = DIAG ? sh.sq[i] * d : sh.sq[i];
        sh.pvc[tid] = make_float4(kd, qd, d, beta * sh.sk[i]);
        kq = sh.sq[i] * sh.sk[i];
    }
    if (tid < 128) {
        const int x = tid;
        int bw;
        const int p = slot_row(hi, x, bw);
        float av = 0.f, al = 0.f;
        if (p >= 0) {
            const int wi = bw == 8 ? 0 : (bw == 4 ? 1 : 2);
            const int i = sh.sperm[p];
            const float r = sh.sr[p];
            const float ki = sh.sk[i], qi = sh.sq[i];
            const float di = DIAG ? sh.sd[i] : 1.0f;
            const float rs = r * lv.fq[wi] * di;
            kt = ki * rs;
            qt = qi * rs;
            const float sc = SCALED ? (bw == 8 ? 1.0f / 256.0f : (bw == 4 ? (1.0f / 14.0f) : 0.5f)) : 1.0f;
            av = beta * ki * (lv.iq[wi] * sc) * __builtin_amdgcn_rcpf(r);
            al = di * (bw == 8 ? sc : (bw == 4 ? (1.0f / 16.0f) * sc : (1.0f / 64.0f) * sc));
            kq += qi * ki;
        }
        sh.av[x] = av;
        if constexpr (DIAG) sh.al[x] = al;
        // the table slots and pivot rows live in wavefronts 0 and 1 only:
        // the others skip the reductions
        kq = wave_sum(kq);
        const float mk = wave_max(fabsf(kt)), mq = wave_max(fabsf(qt));
        if ((tid & 63) == 0) {
            sh.kap[tid >> 6] = kq;
            sh.wmx[tid >> 6] = make_float2(mk, mq);
        }
    }
    __syncthreads();
    const float2 w0 = sh.wmx[0], w1 = sh.wmx[1];
    ek = __builtin_amdgcn_readfirstlane(weight_scale_exp(fmaxf(w0.x, w1.x)));
    eq = __builtin_amdgcn_readfirstlane(weight_scale_exp(fmaxf(w0.y, w1.y)));
    const float kappa = sh.kap[0] + sh.kap[1];
    if (tid < 128) {
        constexpr int X4 = 8 * M8, X2 = 8 * M8 + 16 * M4;
        const int x = tid;
        int slice, ridx;
        if (x < X4) {
            slice = x & 7;
            ridx = x >> 3;
        } else if (x < X2) {
            const int c = (x - X4) >> 1;
            slice = c & 7;
            ridx = M8 + 2 * (c >> 3) + ((x - X4) & 1);
        } else {
            const int c = (x - X2) >> 2;
            slice = c & 7;
            ridx = M8 + 2 * M4 + 4 * (c >> 3) + ((x - X2) & 3);
        }
        const float ks = __builtin_amdgcn_ldexpf(kt, ek), qs = __builtin_amdgcn_ldexpf(qt, eq);
        const _Float16 kh = static_cast<_Float16>(ks), qh = static_cast<_Float16>(qs);
        const _Float16 kl = static_cast<_Float16>(ks - static_cast<float>(kh));
        const _Float16 ql = static_cast<_Float16>(qs - static_cast<float>(qh));
        _Float16(&dst)[4][4] = sh.aop[slice][ridx >> 2];
        dst[0][ridx & 3] = kh;
        dst[1][ridx & 3] = kl;
        dst[2][ridx & 3] = qh;
        dst[3][ridx & 3] = ql;
    }
    return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(kappa)));
}

// Column sums of the per-thread partials, residual, readout, column factor
// of the code-space update.  cj, vj: column tid's scale and value (threads
// < DV, loaded at the start of the tile).  Ends with a barrier.
template <int DV>
__device__ __forceinline__ void column_sums(const DecodeArgs &a, int tile, float alpha, float beta,
                                            DecodeShared<DV> &sh, float kappa, float cj, float vj);

template <int DV>
__device__ __forceinline__ void column_phase(const DecodeArgs &a, int tile, float alpha, float beta,
                                             DecodeShared<DV> &sh, float kappa, const float (&acK)[4],
                                             const float (&acQ)[4], float cj, float vj)
{
    constexpr int CG = DV / 4;
    const int tid = threadIdx.x;
    sh.red[0][tid / CG][tid % CG] = make_float4(acK[0], acK[1], acK[2], acK[3]);
    sh.red[1][tid / CG][tid % CG] = make_float4(acQ[0], acQ[1], acQ[2], acQ[3]);
    column_sums<DV>(a, tile, alpha, beta, sh, kappa, cj, vj);
}

// The column phase once every thread has written its partials to sh.red.
template <int DV>
__device__ __forceinline__ void column_sums(const DecodeArgs &a, int tile, float alpha, float beta,
                                            DecodeShared<DV> &sh, float kappa, float cj, float vj)
{
    constexpr int NSL = 256 / (DV / 4);
    const int tid = threadIdx.x;
    __syncthreads();
    if (tid < DV) {
        const int j = tid;
        const float *rk = reinterpret_cast<const float *>(&sh.red[0][0][0]);
        const float *rq = reinterpret_cast<const float *>(&sh.red[1][0][0]);
        float sk = rk[j], sq = rq[j];
#pragma unroll
        for (int s = 1; s < NSL; ++s) {
            sk += rk[s * DV + j];
            sq += rq[s * DV + j];
        }
        const float delta = vj - alpha * (cj * sk);     // v - alpha (S^T k)
        a.o[static_cast<size_t>(tile) * DV + j] = alpha * (cj * sq) + beta * kappa * delta;
        sh.bcol[j] = delta * __builtin_amdgcn_rcpf(cj);
    }
    __syncthreads();
}

// Unpack one word's slot-s fields (2^(8-B) q each) and add them, weighted
// by the slot's row constants, to the 4 column partials.
template <int B>
__device__ __forceinline__ void unpack_acc(uint32_t w, const float2 *kq, int x0, float *U, float (&acK)[4],
                                           float (&acQ)[4])
{
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float2 c = kq[x0 + s];
        const uint32_t W = slot_top<B>(w, s);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float u = sbyte(W, e);
            U[4 * s + e] = u;
            acK[e] = fmaf(c.x, u, acK[e]);
            acQ[e] = fmaf(c.y, u, acQ[e]);
        }
    }
}

template <int B>
__device__ __forceinline__ void unpack_word(uint32_t w, float *U)
{
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const uint32_t W = slot_top<B>(w, s);
#pragma unroll
        for (int e = 0; e < 4; ++e) U[4 * s + e] = sbyte(W, e);
    }
}

// ---- codes kept as binary16 between the passes (exact: |2^(8-B) q| <= 127)

// a * h + c with h the low (HI = 0) or high (HI = 1) f16 half of hp, in fp32
// (v_fma_mix_f32: the half is widened exactly inside the FMA).
template <int HI>
__device__ __forceinline__ float fma_mix(float a, uint32_t hp, float c)
{
    float r;
    if constexpr (HI)
        asm("v_fma_mix_f32 %0, %1, %2, %3 op_sel:[0,1,0] op_sel_hi:[0,1,0]" : "=v"(r) : "v"(a), "v"(hp), "v"(c));
    else
        asm("v_fma_mix_f32 %0, %1, %2, %3 op_sel_hi:[0,1,0]" : "=v"(r) : "v"(a), "v"(hp), "v"(c));
    return r;
}

// ---- row-pair layout of the uniform bodies' matrix-core path: register
// Ub[e][g][h] holds column e of rows 4g + 2h (low half) and 4g + 2h + 1
// (high half) of the thread's 16 rows, i.e. half of the B operand of the
// 4x4x4 block for column e and row group g.

typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Byte E of lo_w and of hi_w, read as signed, to an f16 pair (exact).
template <int E>
__device__ __forceinline__ uint32_t sbyte_pair_f16(uint32_t lo_w, uint32_t hi_w)
{
    uint32_t r;
    asm("v_cvt_f16_i16_sdwa %0, sext(%1) dst_sel:WORD_0 dst_unused:UNUSED_PAD src0_sel:BYTE_%c2"
        : "=v"(r) : "v"(lo_w), "i"(E));
    asm("v_cvt_f16_i16_sdwa %0, sext(%1) dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:BYTE_%c2"
        : "+v"(r) : "v"(hi_w), "i"(E));
    return r;
}

// v_mfma_f32_4x4x4_16b_f16: 16 independent 4x4x4 products, block b on
// lanes 4b .. 4b+3.  Lane 4b+i supplies row i of A (4 values along k),
// lane 4b+j column j of B (4 values along k) and receives column j of
// D = A B + C (4 values along i).
__device__ __forceinline__ f32x4 mfma4x4x4(u32x2 a, uint32_t b0, uint32_t b1, f32x4 c)
{
    const u32x2 b{b0, b1};
    return __builtin_amdgcn_mfma_f32_4x4x4f16(__builtin_bit_cast(f16x4, a), __builtin_bit_cast(f16x4, b), c, 0, 0,
                                              0);
}

// The thread's 16 rows (8-bit words, then the slots of the 4-bit and 2-bit
// words) as row-pair f16 registers.
template <int M8, int M4, int M2>
__device__ __forceinline__ void unpack_row_pairs(const uint32_t (&w)[M8 + M4 + M2], uint32_t (&Ub)[4][4][2])
{
    static_assert(M8 + 2 * M4 + 4 * M2 == 16, "16 rows per thread");
    static_assert(M8 % 4 == 0 && M4 % 2 == 0, "row groups of 4 hold rows of one width");
    constexpr int G4 = M8 / 4, G2 = (M8 + 2 * M4) / 4;    // first row group of the 4- and 2-bit rows
#pragma unroll
    for (int g = 0; g < G4; ++g)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint32_t lo = w[4 * g + 2 * h], hi = w[4 * g + 2 * h + 1];
            Ub[0][g][h] = sbyte_pair_f16<0>(lo, hi);
            Ub[1][g][h] = sbyte_pair_f16<1>(lo, hi);
            Ub[2][g][h] = sbyte_pair_f16<2>(lo, hi);
            Ub[3][g][h] = sbyte_pair_f16<3>(lo, hi);
        }
#pragma unroll
    for (int m = 0; m < M4; ++m) {
        const uint32_t s0 = slot_top<4>(w[M8 + m], 0), s1 = slot_top<4>(w[M8 + m], 1);
        const int g = G4 + m / 2, h = m & 1;
        Ub[0][g][h] = sbyte_pair_f16<0>(s0, s1);
        Ub[1][g][h] = sbyte_pair_f16<1>(s0, s1);
        Ub[2][g][h] = sbyte_pair_f16<2>(s0, s1);
        Ub[3][g][h] = sbyte_pair_f16<3>(s0, s1);
    }
#pragma unroll
    for (int m = 0; m < M2; ++m) {
        const uint32_t wm = w[M8 + M4 + m];
        const int g = G2 + m;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint32_t s0 = slot_top<2>(wm, 2 * h), s1 = slot_top<2>(wm, 2 * h + 1);
            Ub[0][g][h] = sbyte_pair_f16<0>(s0, s1);
            Ub[1][g][h] = sbyte_pair_f16<1>(s0, s1);
            Ub[2][g][h] = sbyte_pair_f16<2>(s0, s1);
            Ub[3][g][h] = sbyte_pair_f16<3>(s0, s1);
        }
    }
    // The converts are inline assembly, whose register writes the compiler's
    // hazard checks do not see, and the matrix core reads these registers
    // later.  An s_nop tied to every one of them comes after the last
    // convert and before any read, whatever the schedule, and keeps the wait
    // states a VALU write needs before a matrix-core read.
    asm volatile("s_nop 4"
                 : "+v"(Ub[0][0][0]), "+v"(Ub[0][0][1]), "+v"(Ub[0][1][0]), "+v"(Ub[0][1][1]), "+v"(Ub[0][2][0]),
                   "+v"(Ub[0][2][1]), "+v"(Ub[0][3][0]), "+v"(Ub[0][3][1]), "+v"(Ub[1][0][0]), "+v"(Ub[1][0][1]),
                   "+v"(Ub[1][1][0]), "+v"(Ub[1][1][1]), "+v"(Ub[1][2][0]), "+v"(Ub[1][2][1]), "+v"(Ub[1][3][0]),
                   "+v"(Ub[1][3][1]), "+v"(Ub[2][0][0]), "+v"(Ub[2][0][1]), "+v"(Ub[2][1][0]), "+v"(Ub[2][1][1]),
                   "+v"(Ub[2][2][0]), "+v"(Ub[2][2][1]), "+v"(Ub[2][3][0]), "+v"(Ub[2][3][1]), "+v"(Ub[3][0][0]),
                   "+v"(Ub[3][0][1]), "+v"(Ub[3][1][0]), "+v"(Ub[3][1][1]), "+v"(Ub[3][2][0]), "+v"(Ub[3][2][1]),
                   "+v"(Ub[3][3][0]), "+v"(Ub[3][3][1]));
}

// The thread's column partials of S^T k and S^T q (before the c_j factor)
// from 16 4x4x4 products, written to sh.red for the column phase.  The
// operand table of row_constants_mfma must be complete (a barrier after
// it).  The 4 threads of a block share their rows and own 4 different
// column words; thread type cg & 3 supplies weight type cg & 3.
__device__ __forceinline__ void matvec_partials(DecodeShared<128> &sh, int slice, int cg,
                                                const uint32_t (&Ub)[4][4][2], int ek, int eq)
{
    u32x2 A[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) A[g] = *reinterpret_cast<const u32x2 *>(&sh.aop[slice][g][cg & 3][0]);
    float *redK = &sh.red[0][slice][cg].x, *redQ = &sh.red[1][slice][cg].x;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        f32x4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int g = 0; g < 4; ++g) d = mfma4x4x4(A[g], Ub[e][g][0], Ub[e][g][1], d);
        redK[e] = __builtin_amdgcn_ldexpf(d[0] + d[1], -ek);    // the column partials go straight to LDS
        redQ[e] = __builtin_amdgcn_ldexpf(d[2] + d[3], -eq);
        __builtin_amdgcn_sched_barrier(0);    // one column's chain at a time: 4 accumulators live
    }
}

// ---- row-mix heads (compact layout, 8- and 4-bit rows in any split, d_v =
// 128).  Word m of thread (slice, cg) is row group g = slice + 8 m.  A block's
// K dimension is 4 consecutive words of one slice (word group j = m / 4)
// read through slot view s: s = 0 the 8-bit row or slot 0 of a 4-bit
// group, s = 1 slot 1 of a 4-bit group.

// The A operands of the row-mix blocks from the row-table weights that
// row_constants left in sh.kq, prescaled by 2^ek and 2^eq as in
// row_constants_mfma: aopv[slice][j][s][type][m mod 4].  Views that hold no
// row (slot 1 of an 8-bit group, an empty 4-bit slot, a group past the
// head's last) get zero weights.  Two barriers; the table is complete
// after the second.
__device__ __forceinline__ void row_operands_rowmix(const HeadInfo &hi, DecodeShared<128> &sh, int &ek, int &eq)
{
    const int tid = threadIdx.x;
    float mk = 0.f, mq = 0.f;
    if (tid < kSlotTable) {
        const float2 c = sh.kq[tid];
        mk = fabsf(c.x);
        mq = fabsf(c.y);
    }
    mk = wave_max(mk);
    mq = wave_max(mq);
    if ((tid & 63) == 0) sh.wmx[tid >> 6] = make_float2(mk, mq);
    __syncthreads();
    const float2 w0 = sh.wmx[0], w1 = sh.wmx[1], w2 = sh.wmx[2];    // the table slots live in wavefronts 0 .. 2
    ek = __builtin_amdgcn_readfirstlane(weight_scale_exp(fmaxf(fmaxf(w0.x, w1.x), w2.x)));
    eq = __builtin_amdgcn_readfirstlane(weight_scale_exp(fmaxf(fmaxf(w0.y, w1.y), w2.y)));
    // one (slice, word, view) entry per thread
    const int slice = tid & 7, m = (tid >> 3) & 15, v = tid >> 7;
    const int g = slice + 8 * m;
    const int g8 = hi.g8;
    int x = -1;
    if (g < g8) x = v == 0 ? g : -1;
    else if (g < static_cast<int>(hi.groups)) x = g8 + 2 * (g - g8) + v;
    const float2 c = x >= 0 ? sh.kq[x] : make_float2(0.f, 0.f);
    const float ks = __builtin_amdgcn_ldexpf(c.x, ek), qs = __builtin_amdgcn_ldexpf(c.y, eq);
    const _Float16 kh = static_cast<_Float16>(ks), qh = static_cast<_Float16>(qs);
    const _Float16 kl = static_cast<_Float16>(ks - static_cast<float>(kh));
    const _Float16 ql = static_cast<_Float16>(qs - static_cast<float>(qh));
    _Float16(&dst)[4][4] = sh.aopv[slice][m >> 2][v];
    dst[0][m & 3] = kh;
    dst[1][m & 3] = kl;
    dst[2][m & 3] = qh;
    dst[3][m & 3] = ql;
    __syncthreads();
}

// One view of a word group: the 4x4x4 block of column E of the thread,
// added to that column's accumulator.  The B operands come from inline
// assembly, whose register writes the compiler's hazard checks do not see,
// and are read by the matrix core right after: the s_nop, tied to them,
// keeps the wait states a VALU write needs before such a read.
template <int E>
__device__ __forceinline__ f32x4 mfma_view(const _Float16 (&A)[4][4], const uint32_t (&v)[4], int cg, f32x4 d)
{
    const u32x2 a = *reinterpret_cast<const u32x2 *>(&A[cg & 3][0]);
    uint32_t b0 = sbyte_pair_f16<E>(v[0], v[1]), b1 = sbyte_pair_f16<E>(v[2], v[3]);
    asm volatile("s_nop 4" : "+v"(b0), "+v"(b1));
    return mfma4x4x4(a, b0, b1, d);
}

// Column E of the row-mix thread's two sums: one chain over the word groups
// and their slot views (one accumulator live), written to LDS unscaled.
// The slot-0 views of the group holding the width boundary (vb) come in
// formed; the other views are formed again for each column rather than kept.
template <int E>
__device__ __forceinline__ void rowmix_column(const DecodeShared<128> &sh, const uint32_t (&w)[16],
                                              const uint32_t (&vb)[4], int slice, int cg, int g8, int ng, int ek,
                                              int eq, float *redK, float *redQ)
{
    f32x4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (32 * j >= ng) break;
        if (32 * j + 32 <= g8) {
            // 8-bit words only: their bytes are the codes
            const uint32_t v[4] = {w[4 * j], w[4 * j + 1], w[4 * j + 2], w[4 * j + 3]};
            d = mfma_view<E>(sh.aopv[slice][j][0], v, cg, d);
        } else {
            uint32_t v[4];
            if (32 * j >= g8) {
#pragma unroll
                for (int k = 0; k < 4; ++k) v[k] = slot_top<4>(w[4 * j + k], 0);
                d = mfma_view<E>(sh.aopv[slice][j][0], v, cg, d);
            } else {
                d = mfma_view<E>(sh.aopv[slice][j][0], vb, cg, d);    // the group of the width boundary
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) v[k] = slot_top<4>(w[4 * j + k], 1);
            d = mfma_view<E>(sh.aopv[slice][j][1], v, cg, d);
        }
    }
    redK[E] = __builtin_amdgcn_ldexpf(d[0] + d[1], -ek);
    redQ[E] = __builtin_amdgcn_ldexpf(d[2] + d[3], -eq);
    __builtin_amdgcn_sched_barrier(0);
}

// All four columns of the row-mix thread's two sums in one pass over the
// word groups (four accumulators live): each group's slot views are formed
// once rather than once per column.  For bodies whose register peak lies
// after the column phase (the refitting body).
__device__ __forceinline__ void rowmix_columns4(const DecodeShared<128> &sh, const uint32_t (&w)[16], int slice,
                                                int cg, int g8, int ng, int ek, int eq, float *redK, float *redQ)
{
    f32x4 d0 = {0.f, 0.f, 0.f, 0.f}, d1 = d0, d2 = d0, d3 = d0;
    auto all = [&](const _Float16 (&A)[4][4], const uint32_t (&v)[4]) {
        d0 = mfma_view<0>(A, v, cg, d0);
        d1 = mfma_view<1>(A, v, cg, d1);
        d2 = mfma_view<2>(A, v, cg, d2);
        d3 = mfma_view<3>(A, v, cg, d3);
    };
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (32 * j >= ng) break;
        if (32 * j + 32 <= g8) {
            const uint32_t v[4] = {w[4 * j], w[4 * j + 1], w[4 * j + 2], w[4 * j + 3]};
            all(sh.aopv[slice][j][0], v);
        } else {
            uint32_t v[4];
            if (32 * j >= g8) {
#pragma unroll
                for (int k = 0; k < 4; ++k) v[k] = slot_top<4>(w[4 * j + k], 0);
                all(sh.aopv[slice][j][0], v);
            } else {
                // the group of the width boundary: 8-bit below g8, slot 0 of a 4-bit group above
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    v[k] = slice + 8 * (4 * j + k) < g8 ? w[4 * j + k] : slot_top<4>(w[4 * j + k], 0);
                all(sh.aopv[slice][j][0], v);
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) v[k] = slot_top<4>(w[4 * j + k], 1);
            all(sh.aopv[slice][j][1], v);
        }
    }
    redK[0] = __builtin_amdgcn_ldexpf(d0[0] + d0[1], -ek);
    redQ[0] = __builtin_amdgcn_ldexpf(d0[2] + d0[3], -eq);
    redK[1] = __builtin_amdgcn_ldexpf(d1[0] + d1[1], -ek);
    redQ[1] = __builtin_amdgcn_ldexpf(d1[2] + d1[3], -eq);
    redK[2] = __builtin_amdgcn_ldexpf(d2[0] + d2[1], -ek);
    redQ[2] = __builtin_amdgcn_ldexpf(d2[2] + d2[3], -eq);
    redK[3] = __builtin_amdgcn_ldexpf(d3[0] + d3[1], -ek);
    redQ[3] = __builtin_amdgcn_ldexpf(d3[2] + d3[3], -eq);
}

// The first half of the row-mix bodies (decode_rowmix and the refitting
// body's refit_rowmix): row constants (divided by the widths' clamp scales
// when SCALED, the form the frozen-scale requantization works in), both sums
// over rows on the matrix cores, the pivot rows' share, and the column
// phase: o is written and delta_j / c_j is left in sh.bcol.  w: the
// thread's 16 code words (0 past the head's last group); pr: its pivot row.
// ALLCOLS: the four columns in one pass (rowmix_columns4), else one at a
// time (fewer registers).
template <bool DIAG, bool SCALED, bool ALLCOLS = false>
__device__ __forceinline__ void rowmix_sums(const DecodeArgs &a, const TileCtx &t, DecodeShared<128> &sh,
                                            const uint32_t (&w)[16], const PivotRegs<128, kCompactPivots> &pr,
                                            const RowColOps &op, int g8, int ng)
{
    const int tid = threadIdx.x;
    const int cg = tid & 31, slice = tid >> 5;
    // v_j waits in LDS for the column phase (c_j is kept there for the pivot
    // rows), so neither is held in registers through the row sums
    if (tid < 128) sh.bcol[tid] = op.v;
    const float kappa = uniform_f(row_constants<DIAG, 128, SCALED>(t.hi, 128, t.alpha, t.beta, op, sh, a.pool.lv));
    int ek, eq;
    row_operands_rowmix(t.hi, sh, ek, eq);

    float *redK = &sh.red[0][slice][cg].x, *redQ = &sh.red[1][slice][cg].x;
    // slot-0 views of the word group holding the width boundary (if any),
    // formed once: there the width changes from one slice to the next
    if constexpr (ALLCOLS) {
        rowmix_columns4(sh, w, slice, cg, g8, ng, ek, eq, redK, redQ);
    } else {
        uint32_t vb[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if ((g8 >> 5) == j && (g8 & 31) != 0) {
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    vb[k] = slice + 8 * (4 * j + k) < g8 ? w[4 * j + k] : slot_top<4>(w[4 * j + k], 0);
            }
        rowmix_column<0>(sh, w, vb, slice, cg, g8, ng, ek, eq, redK, redQ);
        rowmix_column<1>(sh, w, vb, slice, cg, g8, ng, ek, eq, redK, redQ);
        rowmix_column<2>(sh, w, vb, slice, cg, g8, ng, ek, eq, redK, redQ);
        rowmix_column<3>(sh, w, vb, slice, cg, g8, ng, ek, eq, redK, redQ);
    }
    pivot_partials_slice(t, slice, cg, pr, sh);

    column_sums<128>(a, t.tile, DIAG ? 1.0f : t.alpha, t.beta, sh, kappa, sh.cpiv[tid & 127], sh.bcol[tid & 127]);
}

// a * h + c clamped to [0, 1] by the instruction's clamp bit, h the low
// (HI = 0) or high (HI = 1) binary16 half of hp.
template <int HI>
__device__ __forceinline__ float fma_mix_clamp(float a, uint32_t hp, float c)
{
    float r;
    if constexpr (HI)
        asm("v_fma_mix_f32 %0, %1, %2, %3 op_sel:[0,1,0] op_sel_hi:[0,1,0] clamp" : "=v"(r) : "v"(a), "v"(hp), "v"(c));
    else
        asm("v_fma_mix_f32 %0, %1, %2, %3 op_sel_hi:[0,1,0] clamp" : "=v"(r) : "v"(a), "v"(hp), "v"(c));
    return r;
}

// Scale of the clamped form of a B-bit field (requant_field_p): the field
// value y in [1, 2^B - 1] is handled as (y - 1) / S clamped to [0, 1].
// S = 2^B - 2 for 4- and 2-bit fields, where the top of the clamp is the
// top level; S = 256 for 8-bit fields, whose clamp then tops at 257 and
// v_cvt_pk_u8_f32's saturation at 255 does the rest.  2- and 8-bit scales
// are powers of two.
template <int B>
__device__ __forceinline__ constexpr float clamp_scale()
{
    return B == 8 ? 256.0f : static_cast<float>((1 << B) - 2);
}

// New field in byte E of P from the old field in half HALF of hp; the
// arithmetic of requant_word below, with the clamp to [1, 2^B - 1] from the
// FMA's clamp bit: it forms
//     (y - 1) / S = (al / S) U + (a_s / S) bc_j + (2^(B-1) - 1) / S
// (al and a_s arrive divided by S) clamped to [0, 1], and one full-rate FMA
// scales it back; on gfx950 that replaces a half-rate med3.  The scalings
// are exact for 8- and 2-bit fields and cost a few ulp of the field value
// (at most 15) for 4-bit ones.
template <int B, int E, int HALF>
__device__ __forceinline__ uint32_t requant_field_p(uint32_t hp, float al, float a_s, float bce, uint32_t P)
{
    constexpr float S = clamp_scale<B>();
    constexpr float c0 = static_cast<float>((1 << (B - 1)) - 1) / S;
    const float tt = fmaf(a_s, bce, c0);
    const float y01 = fma_mix_clamp<HALF>(al, hp, tt);
    return __builtin_amdgcn_cvt_pk_u8_f32(fmaf(y01, S, 1.0f), E, P);
}

template <int B, int HALF>
__device__ __forceinline__ uint32_t requant_slot_p(const uint32_t (&Ub)[4][4][2], int g, int h, float al, float a_s,
                                                   const float (&bc)[4])
{
    uint32_t P = 0;
    P = requant_field_p<B, 0, HALF>(Ub[0][g][h], al, a_s, bc[0], P);
    P = requant_field_p<B, 1, HALF>(Ub[1][g][h], al, a_s, bc[1], P);
    P = requant_field_p<B, 2, HALF>(Ub[2][g][h], al, a_s, bc[2], P);
    P = requant_field_p<B, 3, HALF>(Ub[3][g][h], al, a_s, bc[3], P);
    return P;
}

// New word of 8/B slots (row-table slots x0 + s, thread rows r0 + s) from
// the row-pair registers; as requant_word otherwise.  av and alt: the row
// constants of row_constants_mfma with SCALED set.  r0 is a constant
// once the caller's loops are unrolled, so every register index folds.
template <int B, bool DIAG>
__device__ __forceinline__ uint32_t requant_word_p(const uint32_t (&Ub)[4][4][2], int r0, const float *av,
                                                   const float *alt, int x0, float al_w, const float (&bc)[4])
{
    constexpr uint32_t flip = B == 8 ? 0x80808080u : (B == 4 ? 0x88888888u : 0xAAAAAAAAu);
    // the fields are handled as (y - 1) / S (requant_field_p): av and the
    // per-row gates come divided by S from the row constants, the scalar
    // gate is divided here
    constexpr float sc = 1.0f / clamp_scale<B>();
    uint32_t out = 0;
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const int r = r0 + s;
        const float a_s = av[x0 + s];
        const float al = DIAG ? alt[x0 + s] : al_w * sc;
        const uint32_t P = (r & 1) ? requant_slot_p<B, 1>(Ub, r >> 2, (r >> 1) & 1, al, a_s, bc)
                                   : requant_slot_p<B, 0>(Ub, r >> 2, (r >> 1) & 1, al, a_s, bc);
        out |= P << (s * B);
    }
    return out ^ flip;
}

// Row r of the thread's 16 (row-pair register layout of unpack_row_pairs):
// its row-table slot (= physical row in a uniform layout) and width.
template <int M8, int M4>
__device__ __forceinline__ constexpr int thread_row_width(int r)
{
    return r < M8 ? 8 : (r < M8 + 2 * M4 ? 4 : 2);
}

template <int M8, int M4>
__device__ __forceinline__ int thread_row_slot(int r, int slice)
{
    constexpr int X4 = 8 * M8, X2 = 8 * M8 + 16 * M4;
    if (r < M8) return slice + 8 * r;
    if (r < M8 + 2 * M4) {
        const int k = r - M8;
        return X4 + 2 * (slice + 8 * (k >> 1)) + (k & 1);
    }
    const int k = r - M8 - 2 * M4;
    return X2 + 4 * (slice + 8 * (k >> 2)) + (k & 3);
}

// ---- the gate term of the refit's unrounded codes on the matrix cores.
// Per field y = al U + av_i bc_j, U the old code as the converts left it.
// A 4x4x4 binary16 block with A = al I (diagonal) and B = the 4 rows'
// codes of a lane's column returns al U + C for those rows.  With al a
// binary16 value the product al U (|U| <= 127) is exact in fp32 and the
// other three products are zero; the block's addition of C is not always
// the correctly rounded one, though: measured on gfx950 it equals the FMA
// when C is of the magnitude of al U and is otherwise within one ulp of it.
// al = alpha 2^(b-8) is a binary16 value when it is zero or a normal
// binary16 number equal to alpha 2^(b-8) (a bf16 gate not far below 1, for
// instance); otherwise the vector-unit FMA is used.  A 4x4x4 block costs the
// SIMD about as much issue time as four vector FMAs (measured), so this pays
// only where it also shortens the vector-unit work (the refitting body,
// which then needs no separate product); the frozen-scale bodies keep the
// gate term on the vector unit.

// Exactly a normal binary16 value (or zero).
__device__ __forceinline__ bool binary16_exact(float x)
{
    const float ax = fabsf(x);
    return static_cast<float>(static_cast<_Float16>(x)) == x && (x == 0.f || (ax >= 0x1p-14f && ax <= 65504.f));
}

// A operand of the diagonal block: lane 4b + i supplies row i of A, al at
// column i and zeros elsewhere.
__device__ __forceinline__ u32x2 diag_operand(float al, int i)
{
    const uint32_t h = __builtin_bit_cast(uint16_t, static_cast<_Float16>(al));
    const uint32_t v = (i & 1) ? (h << 16) : h;
    return (i & 2) ? u32x2{0u, v} : u32x2{v, 0u};
}

// Whether the uniform layout's gate factors alpha, alpha / 16, alpha / 64
// (of the widths it holds) are binary16 values.
template <int M8, int M4, int M2>
__device__ __forceinline__ bool gate_on_matrix_cores(float alpha)
{
    return (M8 == 0 || binary16_exact(alpha)) && (M4 == 0 || binary16_exact(alpha * (1.0f / 16.0f))) &&
           (M2 == 0 || binary16_exact(alpha * (1.0f / 64.0f)));
}

// a * b + c clamped to [0, 1] by the instruction's clamp bit.
__device__ __forceinline__ float fma_clamp(float a, float b, float c)
{
    float r;
    asm("v_fma_f32 %0, %1, %2, %3 clamp" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

// New word from the unpacked old fields: per field
//   y = al U + av_i bc_j + 2^(B-1)        (code + bias, Eq. 3 argument)
// clamped to [1, 2^B - 1] (i.e. code in [-q_b, q_b]), rounded to nearest
// even and packed to a byte by v_cvt_pk_u8_f32, then the bias is removed
// from all fields at once by flipping each field's top bit.  The clamp is
// the FMA's clamp bit on (y - 1) / S, scaled back by one more FMA
// (requant_field_p, clamp_scale): av and the per-row gates alt come
// divided by S (row_constants with SCALED set), the scalar gate al_w is
// divided here.
template <int B, bool DIAG>
__device__ __forceinline__ uint32_t requant_word(const float *U, const float *av, const float *alt, int x0,
                                                 float al_w, const float (&bc)[4])
{
    constexpr float S = clamp_scale<B>();
    constexpr float c0 = static_cast<float>((1 << (B - 1)) - 1) / S;
    constexpr uint32_t flip = B == 8 ? 0x80808080u : (B == 4 ? 0x88888888u : 0xAAAAAAAAu);
    uint32_t out = 0;
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float a_s = av[x0 + s];
        const float al = DIAG ? alt[x0 + s] : al_w * (1.0f / S);
        uint32_t P = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float tt = fmaf(a_s, bc[e], c0);
            const float y01 = fma_clamp(al, U[4 * s + e], tt);
            P = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(y01, S, 1.0f), e, P);
        }
        out |= P << (s * B);
    }
    return out ^ flip;
}


// ---- whole FP16 heads (shared by the frozen-step and refitting launches:
// such a head has no integer rows to fit, so every mode runs this body)

// A head whose every row is an FP16 pivot (d = 128).  Thread (slice, cg)
// holds columns 4 cg .. 4 cg + 3 of rows p = slice + 8 m as two binary16
// pairs; the FMAs read the halves directly (v_fma_mix), so nothing is
// unpacked.  The column phase runs with unit column factors.  Each value
// becomes X = d_i S + beta k_i delta_j rounded to binary16 (nearest even),
// stored in place; r and c are left alone (no integer rows to fit).
template <bool BF16, bool DIAG>
__device__ __forceinline__ void decode_f16head(const DecodeArgs &a, const TileCtx &t, DecodeShared<128> &sh)
{
    const int tid = threadIdx.x;
    const int cg = tid & 31, slice = tid >> 5;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(t.codes, 0, 128 * 256, 0x00020000);
    // one 8-byte access per row and thread: a half-wavefront covers a whole
    // 256-byte row
    u32x2 S[16];
#pragma unroll
    for (int m = 0; m < 16; ++m)
        S[m] = __builtin_amdgcn_raw_buffer_load_b64(rs, (slice + 8 * m) * 256 + 8 * cg, 0, CodeWords::kLoad);
    // k, q, the gate and the permutation by row, v by column (the r and c
    // slots of the record are not read)
    const PoolView &P = a.pool;
    float vj = 0.f;
    int perm = 0;
    if (tid < 128) {
        const size_t off = (static_cast<size_t>(t.b) * P.Hqk + t.hq) * 128 + tid;
        sh.sk[tid] = act_ld<BF16>(a.k, off);
        sh.sq[tid] = act_ld<BF16>(a.q, off);
        if constexpr (DIAG) sh.sd[tid] = act_ld<BF16>(a.alpha, static_cast<size_t>(t.tile) * 128 + tid);
        perm = P.perm[t.h * 128 + tid];
        vj = act_ld<BF16>(a.v, static_cast<size_t>(t.tile) * 128 + tid);
    }
    __syncthreads();
    float kq = 0.f;
    if (tid < 128) {
        // physical row p = tid holds logical row perm[p]
        const int i = perm;
        const float ki = sh.sk[i], qi = sh.sq[i];
        const float di = DIAG ? sh.sd[i] : 1.0f;       // the scalar gate is applied with the columns
        sh.kq[tid] = make_float2(ki * di, qi * di);
        sh.av[tid] = t.beta * ki;
        if constexpr (DIAG) sh.al[tid] = di;
        kq = qi * ki;
    }
    kq = wave_sum(kq);
    if ((tid & 63) == 0) sh.kap[tid >> 6] = kq;
    __syncthreads();
    const float kappa = (sh.kap[0] + sh.kap[1]) + (sh.kap[2] + sh.kap[3]);

    float acK[4] = {0.f, 0.f, 0.f, 0.f}, acQ[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int m = 0; m < 16; ++m) {
        const float2 c = sh.kq[slice + 8 * m];
        acK[0] = fma_mix<0>(c.x, S[m].x, acK[0]);
        acQ[0] = fma_mix<0>(c.y, S[m].x, acQ[0]);
        acK[1] = fma_mix<1>(c.x, S[m].x, acK[1]);
        acQ[1] = fma_mix<1>(c.y, S[m].x, acQ[1]);
        acK[2] = fma_mix<0>(c.x, S[m].y, acK[2]);
        acQ[2] = fma_mix<0>(c.y, S[m].y, acQ[2]);
        acK[3] = fma_mix<1>(c.x, S[m].y, acK[3]);
        acQ[3] = fma_mix<1>(c.y, S[m].y, acQ[3]);
    }
    column_phase<128>(a, t.tile, DIAG ? 1.0f : t.alpha, t.beta, sh, kappa, acK, acQ, 1.0f, vj);
    if (a.f16_c_one && tid < 128) const_cast<float *>(t.cc)[tid] = 1.0f;

    const float4 b4 = *reinterpret_cast<const float4 *>(&sh.bcol[4 * cg]);   // delta_j
    const float dl[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
    for (int m = 0; m < 16; ++m) {
        const int p = slice + 8 * m;
        const float bk = sh.av[p];
        const float dg = DIAG ? sh.al[p] : t.alpha;
        const float x0 = fmaf(bk, dl[0], dg * half_lo(S[m].x)), x1 = fmaf(bk, dl[1], dg * half_hi(S[m].x));
        const float x2 = fmaf(bk, dl[2], dg * half_lo(S[m].y)), x3 = fmaf(bk, dl[3], dg * half_hi(S[m].y));
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{pack_halves(x0, x1), pack_halves(x2, x3)}, rs, p * 256 + 8 * cg, 0,
                                              CodeWords::kStore);
    }
}

template <bool BF16, bool DIAG>
__device__ __forceinline__ void run_f16head(const DecodeArgs &a, TileCtx &t, int slot, DecodeShared<128> &sh)
{
    // the tile record is 128 rows x 128 binary16 values, then the unused r and c
    uint8_t *rec = a.pool.base + static_cast<uint64_t>(slot) * a.pool.slot_bytes + t.off;
    t.codes = reinterpret_cast<uint32_t *>(rec);
    t.rr = reinterpret_cast<const float *>(rec + 128 * 256);
    t.cc = t.rr + 128;
    decode_f16head<BF16, DIAG>(a, t, sh);
}

}  // namespace
}  // namespace stepq
