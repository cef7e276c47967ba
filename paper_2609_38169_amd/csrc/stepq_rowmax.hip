// The decode step with the row-wise absmax requantization of the INT-b
// baseline the paper compares against (Section 5.1): per key row
//     r'_i = max_j |X_ij| (floored at 2^-60),   c'_j = 1,
//     q'_ij = clip(round(X_ij q_b / r'_i), -q_b, q_b)
// (N1; under N2 the levels are 2^(8-b) q and r' divides by the top level,
// which gives the same r' = r max_j |z_ij| / q_b below).
//
// Uniform layouts (d = 128) have a body of their own.  It runs the frozen
// body's first half (unpack, S^T k and S^T q on the matrix cores, residual,
// readout), then works with
//     z_ij = c_j y_ij = (alpha 2^(b-8) c_j) U_ij + (beta k_i q_b / r_i) delta_j,
// the new value X_ij in units of r_i / q_b (U = 2^(8-b) q, the unpacked
// field; y the frozen body's unrounded code on the old scales), kept in
// registers: 64 values per thread, two operations each.  The row maxima
// M_i = max_j |z_ij| meet in LDS (the 32 lanes that share a row first pair
// up), then
//     r'_i = r_i M_i / q_b,   h_i = r_i / r'_i,   q'_ij = round(z_ij h_i),
// one FMA (with the field bias) and the round-and-pack per element.  No
// clamp is needed: |z_ij h_i| <= q_b up to a few ulp, and the biased value
// rounds inside [1, 2^b - 1].  Other layouts take the generic refitting
// body (stepq_refit_body.h).
#include "stepq_refit_body.h"

namespace stepq {
namespace {

struct RowmaxShared {
    DecodeShared<128> d;     // its red[] holds the row maxima' pair partials after the column phase
    float hrow[128];         // h_i = r_i / r'_i by physical row
    float dcol[128];         // delta_j
    float ccol[128];         // c_j
};

// Column phase of the row-absmax body: o, and delta_j, c_j into LDS.
// Ends with a barrier.
__device__ __forceinline__ void column_sums_rowmax(const DecodeArgs &a, int tile, float alpha, float beta,
                                                   RowmaxShared &sh, float kappa, float cj, float vj)
{
    const int tid = threadIdx.x;
    __syncthreads();
    if (tid < 128) {
        const int j = tid;
        const float *rk = reinterpret_cast<const float *>(&sh.d.red[0][0][0]);
        const float *rq = reinterpret_cast<const float *>(&sh.d.red[1][0][0]);
        float sk = rk[j], sq = rq[j];
#pragma unroll
        for (int s = 1; s < 8; ++s) {
            sk += rk[s * 128 + j];
            sq += rq[s * 128 + j];
        }
        const float delta = vj - alpha * (cj * sk);     // v - alpha (S^T k)
        a.o[static_cast<size_t>(tile) * 128 + j] = alpha * (cj * sq) + beta * kappa * delta;
        sh.dcol[j] = delta;
        sh.ccol[j] = cj;
    }
    __syncthreads();
}

// max(|a|, |b|, |c|) in one instruction.  Written out because the
// compiler's own form would first quiet each input (the values come from
// inline assembly, which it cannot prove free of signalling NaNs); finite
// values only reach it here.
__device__ __forceinline__ float max3_abs(float a, float b, float c)
{
    float r;
    asm("v_max3_f32 %0, |%1|, |%2|, |%3|" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

// z of thread row r, column e, from the row-pair registers.
template <bool DIAG>
__device__ __forceinline__ float row_z(uint32_t hp, int half, float coef, float a_s, float delta)
{
    const float tt = a_s * delta;
    return half ? fma_mix<1>(coef, hp, tt) : fma_mix<0>(coef, hp, tt);
}

// Half H (thread rows 8H .. 8H+7) of the row-absmax requantization: z and
// the row maxima over the thread's 4 columns, paired between lanes 2k and
// 2k+1 (non-negative: integer order of the bit patterns is float order)
// and written to part[row][pair]; then one thread per row of the half
// (64 rows) forms M_i, r'_i (stored) and h_i; then the half's words are
// requantized from z.  Two barriers.
template <bool DIAG, int M8, int M4, int M2, int H>
__device__ __forceinline__ void rowmax_half(const TileCtx &t, RowmaxShared &sh, const uint32_t (&Ub)[4][4][2],
                                            float *part, const CodeWords &cw)
{
    const int tid = threadIdx.x;
    const int cg = tid & 31, slice = tid >> 5;
    // delta_j and c_j of the thread's columns, read for each half: they are
    // not held through the other half's reduction
    const float4 d4 = *reinterpret_cast<const float4 *>(&sh.dcol[4 * cg]);
    const float4 c4 = *reinterpret_cast<const float4 *>(&sh.ccol[4 * cg]);
    const float dl[4] = {d4.x, d4.y, d4.z, d4.w};
    const float cl[4] = {c4.x, c4.y, c4.z, c4.w};
    float z[8][4];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const int r = 8 * H + k;
        const int bw = thread_row_width<M8, M4>(r);
        const int x = thread_row_slot<M8, M4>(r, slice);
        const float a_s = sh.d.av[x];
        // alpha 2^(b-8) (the scalar gate), or d_i 2^(b-8) per row (channel-wise)
        const float al = DIAG ? sh.d.al[x] : t.alpha * (bw == 8 ? 1.0f : (bw == 4 ? (1.0f / 16.0f) : (1.0f / 64.0f)));
#pragma unroll
        for (int e = 0; e < 4; ++e)
            z[k][e] = row_z<DIAG>(Ub[e][r >> 2][(r >> 1) & 1], r & 1, al * cl[e], a_s, dl[e]);
        const float mx = max3_abs(max3_abs(z[k][0], z[k][1], z[k][2]), z[k][3], z[k][3]);
        const uint32_t u = __float_as_uint(mx);
        part[x * 16 + (cg >> 1)] = __uint_as_float(max(u, dpp_bits<0xB1, 0xF>(u)));    // quad_perm [1,0,3,2]
        __builtin_amdgcn_sched_barrier(0);    // one row at a time: the z values are the only growing set
    }
    __syncthreads();
    if (tid < 64) {
        // thread row 8H + (tid >> 3) of slice tid & 7
        const int r = 8 * H + (tid >> 3);
        const int p = thread_row_slot<M8, M4>(r, tid & 7);
        const float4 *pp = reinterpret_cast<const float4 *>(&part[p * 16]);
        // half the partials at a time: the other half's z and codes are live
        const float4 v0 = pp[0], v1 = pp[1];
        float Mx = max3_abs(v0.x, v0.y, v0.z);
        Mx = max3_abs(Mx, v0.w, v1.x);
        Mx = max3_abs(Mx, v1.y, v1.z);
        Mx = max3_abs(Mx, v1.w, v1.w);
        __builtin_amdgcn_sched_barrier(0);
        const float4 v2 = pp[2], v3 = pp[3];
        Mx = max3_abs(Mx, v2.x, v2.y);
        Mx = max3_abs(Mx, v2.z, v2.w);
        Mx = max3_abs(Mx, v3.x, v3.y);
        Mx = max3_abs(Mx, v3.z, v3.w);
        const int bw = thread_row_width<M8, M4>(r);
        const float inv_qb = bw == 8 ? (1.0f / 127.0f) : (bw == 4 ? (1.0f / 7.0f) : 1.0f);
        const float ro = sh.d.sr[p];
        const float rn = fmaxf((ro * inv_qb) * Mx, kScaleFloor);
        sh.hrow[p] = ro * __builtin_amdgcn_rcpf(rn);
        const_cast<float *>(t.rr)[p] = rn;
    }
    __syncthreads();
    // q' = round(z h) + bias, rounded and packed by v_cvt_pk_u8_f32; the
    // bias comes off with one XOR per word
#pragma unroll
    for (int k = 0; k < 8;) {
        const int r = 8 * H + k;
        const int bw = thread_row_width<M8, M4>(r);
        const int ns = 8 / bw;                       // rows of this word
        const float bias = bw == 8 ? 128.0f : (bw == 4 ? 8.0f : 2.0f);
        uint32_t out = 0;
#pragma unroll
        for (int s = 0; s < ns; ++s) {
            const float h = sh.hrow[thread_row_slot<M8, M4>(r + s, slice)];
            uint32_t P = 0;
            P = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(z[k + s][0], h, bias), 0, P);
            P = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(z[k + s][1], h, bias), 1, P);
            P = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(z[k + s][2], h, bias), 2, P);
            P = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(z[k + s][3], h, bias), 3, P);
            out |= P << (bw * s);
        }
        // word index of thread row r: 8-bit words hold one row, 4-bit two, 2-bit four
        const int m = r < M8 ? r : (r < M8 + 2 * M4 ? M8 + (r - M8) / 2 : M8 + M4 + (r - M8 - 2 * M4) / 4);
        const uint32_t flip = bw == 8 ? 0x80808080u : (bw == 4 ? 0x88888888u : 0xAAAAAAAAu);
        cw.store_m(tid, m, out ^ flip);
        k += ns;
    }
}

template <bool BF16, bool DIAG, int M8, int M4, int M2>
__device__ __forceinline__ void rowmax_uniform(const DecodeArgs &a, const TileCtx &t, RowmaxShared &sh)
{
    constexpr int M = M8 + M4 + M2;
    const int tid = threadIdx.x;
    const int cg = tid & 31, slice = tid >> 5;
    const CodeWords cw(t.codes, 1024u * M);
    uint32_t w[M];
#pragma unroll
    for (int m = 0; m < M; ++m) w[m] = cw.load_m(tid, m);
    const RowColOps op = load_ops<BF16, DIAG, 128>(a, t.tile, t.b, t.hq, t.h, t.rr, t.cc);
    if (tid < 128) sh.d.sr[tid] = op.r;     // old row factor by physical row, for the new ones
    int ek, eq;
    const float kappa = row_constants_mfma<DIAG, M8, M4, M2, 128>(t.beta, op, sh.d, a.pool.lv, ek, eq);
    uint32_t Ub[4][4][2];
    unpack_row_pairs<M8, M4, M2>(w, Ub);
    __syncthreads();    // operand table written
    matvec_partials(sh.d, slice, cg, Ub, ek, eq);
    column_sums_rowmax(a, t.tile, DIAG ? 1.0f : t.alpha, t.beta, sh, kappa, op.c, op.v);

    // The thread's 16 rows in two halves of 8: each half forms its z,
    // reduces its row maxima and is requantized before the next half's z
    // exist, so at most 32 z values are live
    float *part = reinterpret_cast<float *>(&sh.d.red[0][0][0]);    // [128 rows][16 lane pairs]
    if (tid < 128) const_cast<float *>(t.cc)[tid] = 1.0f;    // c' = 1 (c was read at the start)
    rowmax_half<DIAG, M8, M4, M2, 0>(t, sh, Ub, part, cw);
    rowmax_half<DIAG, M8, M4, M2, 1>(t, sh, Ub, part, cw);
}

template <bool BF16, int LAYOUT, bool DIAG>
__global__ __launch_bounds__(256) void rowmax_kernel(DecodeArgs a)
{
    __shared__ RowmaxShared sh;
    constexpr UniformLayout u = kUniformLayouts[LAYOUT - 1];
    constexpr uint32_t r_off = 1024u * (u.m8 + u.m4 + u.m2);
    TileCtx t;
    tile_of(a, r_off + 1024u, t);
    const int slot = a.slot_ids[t.b];
    t.alpha = DIAG ? 1.0f : act_ld<BF16>(a.alpha, t.tile);
    t.beta = act_ld<BF16>(a.beta, t.tile);
    uint8_t *rec = a.pool.base + static_cast<uint64_t>(slot) * a.pool.slot_bytes + t.off;
    t.codes = reinterpret_cast<uint32_t *>(rec);
    t.rr = reinterpret_cast<const float *>(rec + r_off);
    t.cc = t.rr + 128;
    rowmax_uniform<BF16, DIAG, u.m8, u.m4, u.m2>(a, t, sh);
}

template <bool BF16, bool DIAG>
hipError_t launch_rowmax_uniform(const DecodeArgs &a, int layout, unsigned grid, hipStream_t s)
{
    switch (layout) {
    case 1: hipLaunchKernelGGL((rowmax_kernel<BF16, 1, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((rowmax_kernel<BF16, 2, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((rowmax_kernel<BF16, 3, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((rowmax_kernel<BF16, 4, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((rowmax_kernel<BF16, 5, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_rowmax(const DecodeArgs &a, bool bf16, bool diag, int pool_layout, hipStream_t stream)
{
    if (a.pool.dv == 128 && pool_layout >= 1 && pool_layout <= kNumUniformLayouts) {
        const unsigned grid = static_cast<unsigned>(a.batch) * static_cast<unsigned>(a.n_heads);
        if (grid == 0) return hipSuccess;
        if (bf16) return diag ? launch_rowmax_uniform<true, true>(a, pool_layout, grid, stream)
                              : launch_rowmax_uniform<true, false>(a, pool_layout, grid, stream);
        return diag ? launch_rowmax_uniform<false, true>(a, pool_layout, grid, stream)
                    : launch_rowmax_uniform<false, false>(a, pool_layout, grid, stream);
    }
    return launch_refit_mode<Refit::RowAbsmax>(a, bf16, diag, pool_layout, stream);
}

}  // namespace stepq
