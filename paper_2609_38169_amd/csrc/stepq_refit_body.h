// Decode step with a scale refit fused in: the online Key-Row-Aware Dual-Axis refit
// (paper: Section 4.3 row and column factors, the fixed-code column update
// of Appendix C.1, Table C2 steps 4-6).  One 256-thread workgroup per
// (request, value head) tile, as in the frozen-scale kernel, and the same
// first half: unpack, S^T k and S^T q, residual, readout.
//
// Working unit.  Per element the frozen-scale body forms the unrounded new
// code on the old scales,
//     y_ij = X_ij q_b / (r_i c_j).
// Every quantity of the refit is a row or column rescaling of y, so the tile
// is still never formed in real units:
//     m_i   = (r_i / (q_b d_v)) sum_j c_j |y_ij|       r'_i = (m_i / w_i)^(1/2)
//     yh_ij = y_ij r_i / r'_i                         (= X_ij q_b / (r'_i c_j))
//     c0_j  = c_j max_i |yh_ij| / q_b                 (absmax start)
//     z_ij  = round(yh_ij c_j / c0_j)                 (fixed codes; |.| <= q_b)
//     c'_j  = c_j sum_i W_i z_ij yh_ij / sum_i W_i z_ij^2,   W_i = (w_i r'_i / q_b)^2
//     q'_ij = clip(round(yh_ij c_j / c'_j), -q_b, q_b)
// Four passes over the thread's values with three LDS reductions between
// them: row sums (over the lanes that share a row), column maxima (kept per
// width in the thread, so that the scaling by 1/q_b happens once per column
// and thread), and the column sums of the least-squares numerator and
// denominator.  The new r' and c' overwrite the tile's scales; a zero
// denominator keeps c_j.
//
// The generic body also runs the single-axis baseline the paper compares
// against (Section 5.1: symmetric row-wise absmax INT-b): every step
//     r'_i = max_j |X_ij| = (r_i / q_b) max_j c_j |y_ij|,   c'_j = 1,
//     q'_ij = clip(round(y_ij c_j r_i / r'_i), -q_b, q_b),
// i.e. pass 1 with a row maximum instead of a row sum, then pass 4; the
// uniform layouts have a lean body of their own for it (stepq_rowmax.hip).
#pragma once

#include "stepq_device.h"

#include <type_traits>

namespace stepq {
namespace {

constexpr float kScaleFloor = 0x1p-60f;
constexpr float kRoundMagic = 0x1.8p+23f;     // 1.5 2^23: x + this rounds x to an integer (|x| < 2^22)

enum class Refit : int {
    DualAxis = 0,    // Key-Row-Aware Dual-Axis fit (Section 4.3, Appendix C.1)
    RowAbsmax = 1,   // row-wise absmax, column factors 1 (the INT-b baseline)
};

template <int DV>
struct RefitShared {
    DecodeShared<DV> d;
    union {
        float rowp[kSlotTable][DV / 8];            // partials of sum_j c_j |y_ij| by row slot, per column-lane pair
        float4 cmax[256 / (DV / 4)][DV / 4];       // per slice column maxima of |yh| / q_b
    } u;
    float hrow[kSlotTable];                        // r_i / r'_i by row slot (0 for empty slots)
    float wrow[kSlotTable];                        // W_i by row slot
    float wphys[kMaxDk];                           // w by physical row
    float ccol[DV];                                // previous c_j
    float ecol[DV];                                // c_j / c0_j
    float gcol[DV];                                // c_j / c'_j
};

// One row partial of a thread (4 columns of one row slot), combined with
// that of the neighbouring lane (the next 4 columns of the same row) before
// it goes to LDS: sums for the dual-axis fit, maxima (of non-negative
// values) for the row absmax.  Both lanes of a pair write the same value.
template <int DV, Refit MODE>
__device__ __forceinline__ void put_row_partial(RefitShared<DV> &sh, int x, int cg, float acc)
{
    if constexpr (MODE == Refit::DualAxis) acc += dpp_term<0xB1, 0xF>(acc);    // quad_perm [1,0,3,2]
    else acc = __uint_as_float(max(__float_as_uint(acc), dpp_bits<0xB1, 0xF>(__float_as_uint(acc))));
    sh.u.rowp[x][cg >> 1] = acc;
}

// Row partial over the thread's 4 columns: sum_e c_e |y_e| (dual axis) or
// max_e c_e |y_e| (row absmax).
template <Refit MODE>
__device__ __forceinline__ float row_partial(const float *y, const float (&cc)[4])
{
    if constexpr (MODE == Refit::DualAxis) {
        float acc = fabsf(y[0]) * cc[0];
        acc = fmaf(fabsf(y[1]), cc[1], acc);
        acc = fmaf(fabsf(y[2]), cc[2], acc);
        return fmaf(fabsf(y[3]), cc[3], acc);
    } else {
        return fmaxf(fmaxf(fabsf(y[0]) * cc[0], fabsf(y[1]) * cc[1]), fmaxf(fabsf(y[2]) * cc[2], fabsf(y[3]) * cc[3]));
    }
}

// Row slot x (physical row p, width bw, old scale r_p): r' from the lane
// partials, written to the tile; h and W to LDS.  The partials are sums (or
// maxima) of c_j |y_ij| with y = X / (r c nu), nu the width's level step:
// the mean |X_ij| is r nu sum / d_v, W = (w r' nu)^2, and the row-absmax
// factor r' = r max / q_b puts the row's largest entry on the top level in
// either normalisation.  The row and column
// factors are formed with the hardware reciprocal and square root (about one
// ulp each): every later step uses the stored fp32 values, so the codes stay
// consistent with them.
template <int DV, Refit MODE>
__device__ __forceinline__ void refit_row(RefitShared<DV> &sh, int x, int p, int bw, float r_p, float *rr_out,
                                          const LevelTable &lv)
{
    const float iq = bw == 8 ? (1.0f / 127.0f) : (bw == 4 ? (1.0f / 7.0f) : 1.0f);     // 1 / q_b
    const float nu = lv.nu[bw == 8 ? 0 : (bw == 4 ? 1 : 2)];
    if constexpr (MODE == Refit::RowAbsmax) {
        float mx = 0.f;
#pragma unroll
        for (int l = 0; l < DV / 8; l += 4) {
            const float4 v4 = *reinterpret_cast<const float4 *>(&sh.u.rowp[x][l]);
            mx = fmaxf(mx, fmaxf(fmaxf(v4.x, v4.y), fmaxf(v4.z, v4.w)));
        }
        const float rn = fmaxf((r_p * iq) * mx, kScaleFloor);
        sh.hrow[x] = r_p * __builtin_amdgcn_rcpf(rn);
        rr_out[p] = rn;
        return;
    }
    float sum = 0.f;
#pragma unroll
    for (int l = 0; l < DV / 8; l += 4) {
        const float4 v4 = *reinterpret_cast<const float4 *>(&sh.u.rowp[x][l]);
        sum += (v4.x + v4.y) + (v4.z + v4.w);
    }
    const float m = (r_p * nu) * (sum * (1.0f / static_cast<float>(DV)));
    const float w = sh.wphys[p];
    const float rn = fmaxf(__builtin_amdgcn_sqrtf(m * __builtin_amdgcn_rcpf(w)), kScaleFloor);
    sh.hrow[x] = r_p * __builtin_amdgcn_rcpf(rn);
    const float t = (w * rn) * nu;
    sh.wrow[x] = t * t;
    rr_out[p] = rn;
}

// Per-thread column maxima of |yh| kept per width, divided by q_b once.
__device__ __forceinline__ float4 width_max(const float (&m8)[4], const float (&m4)[4], const float (&m2)[4])
{
    float r[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = fmaxf(fmaxf(m8[e] * (1.0f / 127.0f), m4[e] * (1.0f / 7.0f)), m2[e]);
    return make_float4(r[0], r[1], r[2], r[3]);
}

// Column j: absmax start c0_j from the slice maxima; e_j = c_j / c0_j.
template <int DV>
__device__ __forceinline__ void refit_colmax(RefitShared<DV> &sh, int j)
{
    constexpr int NSL = 256 / (DV / 4);
    const float *mx = reinterpret_cast<const float *>(&sh.u.cmax[0][0]);
    float M = 0.f;
#pragma unroll
    for (int s = 0; s < NSL; ++s) M = fmaxf(M, mx[s * DV + j]);
    const float cj = sh.ccol[j];
    const float c0 = fmaxf(cj * M, kScaleFloor);
    sh.ecol[j] = M > 0.f ? cj * __builtin_amdgcn_rcpf(c0) : 0.f;
}

// Column j: the least-squares column factor from the slice sums in d.red.
template <int DV>
__device__ __forceinline__ void refit_colfit(RefitShared<DV> &sh, int j, float *cc_out)
{
    constexpr int NSL = 256 / (DV / 4);
    const float *rn = reinterpret_cast<const float *>(&sh.d.red[0][0][0]);
    const float *rd = reinterpret_cast<const float *>(&sh.d.red[1][0][0]);
    float num = rn[j], den = rd[j];
#pragma unroll
    for (int s = 1; s < NSL; ++s) {
        num += rn[s * DV + j];
        den += rd[s * DV + j];
    }
    const float cj = sh.ccol[j];
    // num / den as a full division: den may be tiny for very small states
    const float cn = den > 0.f ? fmaxf(cj * (num / den), kScaleFloor) : cj;
    sh.gcol[j] = cj * __builtin_amdgcn_rcpf(cn);
    cc_out[j] = cn;
}

// ---- per-word passes on values held in registers (4 columns x 8/B rows)

// y of a word from the row-pair registers of the matrix-core path; the row
// partial sum_e c_e |y| (or max) of each slot goes to LDS.  Slot s of the
// word is thread row r0 + s (a constant once the caller's loops unroll).
template <int B, bool DIAG, Refit MODE>
__device__ __forceinline__ void word_y_p(const uint32_t (&Ub)[4][4][2], int r0, RefitShared<128> &sh, int x0, int cg,
                                         float al_w, const float (&bc)[4], const float (&cc)[4], float *Y)
{
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const int r = r0 + s, g = r >> 2, h = (r >> 1) & 1;
        const float a_s = sh.d.av[x0 + s];
        const float al = DIAG ? sh.d.al[x0 + s] : al_w;
        float *y = Y + 4 * s;
        if (r & 1) {
            y[0] = fma_mix<1>(al, Ub[0][g][h], a_s * bc[0]);
            y[1] = fma_mix<1>(al, Ub[1][g][h], a_s * bc[1]);
            y[2] = fma_mix<1>(al, Ub[2][g][h], a_s * bc[2]);
            y[3] = fma_mix<1>(al, Ub[3][g][h], a_s * bc[3]);
        } else {
            y[0] = fma_mix<0>(al, Ub[0][g][h], a_s * bc[0]);
            y[1] = fma_mix<0>(al, Ub[1][g][h], a_s * bc[1]);
            y[2] = fma_mix<0>(al, Ub[2][g][h], a_s * bc[2]);
            y[3] = fma_mix<0>(al, Ub[3][g][h], a_s * bc[3]);
        }
        put_row_partial<128, MODE>(sh, x0 + s, cg, row_partial<MODE>(y, cc));
    }
}

// Pass 1 of a uniform body with the gate term of y on the matrix cores
// (gate_on_matrix_cores must hold): per row group g and column e, one
// diagonal 4x4x4 block gives y = al U + (av_i bc_j) for the group's 4 rows
// (within one ulp of word_y_p's FMA); Y[4 r + e] for thread row r, and the
// row partials to LDS.
template <int M8, int M4, int M2, Refit MODE>
__device__ __forceinline__ void refit_y_mfma(const uint32_t (&Ub)[4][4][2], RefitShared<128> &sh, int tid, int slice,
                                             int cg, float alpha, const float (&bc)[4], const float (&cc)[4],
                                             float (&Y)[64])
{
    constexpr int G4 = M8 / 4, G2 = (M8 + 2 * M4) / 4;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const float al = g < G4 ? alpha : (g < G2 ? alpha * (1.0f / 16.0f) : alpha * (1.0f / 64.0f));
        const u32x2 A = diag_operand(al, tid & 3);
        float as[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) as[k] = sh.d.av[thread_row_slot<M8, M4>(4 * g + k, slice)];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const f32x4 d = mfma4x4x4(A, Ub[e][g][0], Ub[e][g][1],
                                      f32x4{as[0] * bc[e], as[1] * bc[e], as[2] * bc[e], as[3] * bc[e]});
#pragma unroll
            for (int k = 0; k < 4; ++k) Y[4 * (4 * g + k) + e] = d[k];
        }
#pragma unroll
        for (int k = 0; k < 4; ++k)
            put_row_partial<128, MODE>(sh, thread_row_slot<M8, M4>(4 * g + k, slice), cg,
                                 row_partial<MODE>(&Y[4 * (4 * g + k)], cc));
    }
}

template <int B>
__device__ __forceinline__ void word_scale(float *Y, const float *hrow, int x0)
{
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float h = hrow[x0 + s];
#pragma unroll
        for (int e = 0; e < 4; ++e) Y[4 * s + e] *= h;
    }
}

template <int B>
__device__ __forceinline__ void word_scale_max(float *Y, const float *hrow, int x0, float (&mx)[4])
{
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float h = hrow[x0 + s];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            Y[4 * s + e] *= h;
            mx[e] = fmaxf(mx[e], fabsf(Y[4 * s + e]));
        }
    }
}

template <int B>
__device__ __forceinline__ void word_fit(const float *Y, const float *wrow, int x0, const float (&ec)[4],
                                         float (&num)[4], float (&den)[4])
{
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float W = wrow[x0 + s];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float yh = Y[4 * s + e];
            // round to nearest even by the fp32 grid at 1.5 2^23 (|z| <= q_b):
            // one rounding of the exact product, in two full-rate operations
            const float z = fmaf(yh, ec[e], kRoundMagic) - kRoundMagic;
            const float u = W * z;
            num[e] = fmaf(u, yh, num[e]);
            den[e] = fmaf(u, z, den[e]);
        }
    }
}

// New word: per field round(yh g_j) clamped to +-q_b, packed with a bias of
// 2^(B-1) that the final XOR removes (as in the frozen-scale requantizer).
template <int B>
__device__ __forceinline__ uint32_t word_requant(const float *Y, const float (&g)[4])
{
    constexpr float bias = static_cast<float>(1 << (B - 1));
    constexpr float top = static_cast<float>((1 << B) - 1);
    constexpr uint32_t flip = B == 8 ? 0x80808080u : (B == 4 ? 0x88888888u : 0xAAAAAAAAu);
    uint32_t out = 0;
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        uint32_t P = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float y = fmaf(Y[4 * s + e], g[e], bias);
            y = __builtin_amdgcn_fmed3f(y, 1.0f, top);
            P = __builtin_amdgcn_cvt_pk_u8_f32(y, e, P);
        }
        out |= P << (s * B);
    }
    return out ^ flip;
}

__device__ __forceinline__ void ld4(const float *p, float (&v)[4])
{
    const float4 t = *reinterpret_cast<const float4 *>(p);
    v[0] = t.x;
    v[1] = t.y;
    v[2] = t.z;
    v[3] = t.w;
}

// Uniform layouts at d_v = 128: widths known at compile time, all 64 values
// of the thread kept in registers across the four passes.  PIV: a padded
// pivot head (up to kCompactPivots FP16 pivot rows beside the padded mix,
// t.hi from the head list): its pivot rows join the sums over rows and are
// updated in binary16, and take no part in the fits; the padded mix's empty
// slots (zero codes, no row) get h = W = 0, so they add nothing to the fits
// and keep zero codes.
template <bool BF16, bool DIAG, int M8, int M4, int M2, Refit MODE, bool PIV = false>
__device__ __forceinline__ void refit_uniform(const DecodeArgs &a, const TileCtx &t, RefitShared<128> &sh)
{
    // uniform layouts take the lean row-absmax body of stepq_rowmax.hip
    static_assert(MODE == Refit::DualAxis, "the uniform refitting body runs the dual-axis fit");
    constexpr int M = M8 + M4 + M2;
    constexpr int NE = 4 * (M8 + 2 * M4 + 4 * M2);
    constexpr int X4 = 8 * M8, X2 = 8 * M8 + 16 * M4;
    constexpr int Y4 = 4 * M8, Y2 = 4 * M8 + 8 * M4;     // value offsets of the 4- and 2-bit words
    const int tid = threadIdx.x;
    const int cg = tid & 31, slice = tid >> 5;
    float *rr_out = const_cast<float *>(t.rr);
    float *cc_out = const_cast<float *>(t.cc);
    const CodeWords cw(t.codes, 1024u * M);
    uint32_t w[M];
#pragma unroll
    for (int m = 0; m < M; ++m) w[m] = cw.load_m(tid, m);
    PivotRegs<128, kCompactPivots> pr;
    if constexpr (PIV) pivot_load<128, kCompactPivots>(t, slice, cg, pr);

    const RowColOps op = load_ops<BF16, DIAG, 128>(a, t.tile, t.b, t.hq, t.h, t.rr, t.cc);
    if (tid < 128) {
        sh.ccol[tid] = op.c;
        sh.wphys[tid] = a.pool.roww[t.h * 128 + tid];
    }
    // S^T k and S^T q on the matrix cores, as in the frozen-scale body
    int ek, eq;
    float kappa;
    if constexpr (PIV)
        kappa = row_constants_mfma_piv<DIAG, M8, M4, M2, 128>(t.hi, t.alpha, t.beta, op, sh.d, a.pool.lv, ek, eq);
    else
        kappa = row_constants_mfma<DIAG, M8, M4, M2, 128>(t.beta, op, sh.d, a.pool.lv, ek, eq);
    uint32_t Ub[4][4][2];
    unpack_row_pairs<M8, M4, M2>(w, Ub);
    __syncthreads();    // operand table written
    matvec_partials(sh.d, slice, cg, Ub, ek, eq);
    if constexpr (PIV) pivot_partials_slice(t, slice, cg, pr, sh.d);

    column_sums<128>(a, t.tile, DIAG ? 1.0f : t.alpha, t.beta, sh.d, kappa, op.c, op.v);

    // pass 1: y on the old scales and the row partials
    float bc[4], cc[4];
    ld4(&sh.d.bcol[4 * cg], bc);
    ld4(&sh.ccol[4 * cg], cc);
    if constexpr (PIV) pivot_update<128, kCompactPivots>(t, slice, cg, pr, sh.d, bc);
    float Y[NE];
    bool y_done = false;
    if constexpr (!DIAG) {
        if (gate_on_matrix_cores<M8, M4, M2>(t.alpha)) {
            refit_y_mfma<M8, M4, M2, MODE>(Ub, sh, tid, slice, cg, t.alpha, bc, cc, Y);
            y_done = true;
        }
    }
    if (!y_done) {
#pragma unroll
        for (int m = 0; m < M8; ++m)
            word_y_p<8, DIAG, MODE>(Ub, m, sh, slice + 8 * m, cg, t.alpha, bc, cc, &Y[4 * m]);
#pragma unroll
        for (int m = 0; m < M4; ++m)
            word_y_p<4, DIAG, MODE>(Ub, M8 + 2 * m, sh, X4 + 2 * (slice + 8 * m), cg, t.alpha * (1.0f / 16.0f), bc,
                                    cc, &Y[Y4 + 8 * m]);
#pragma unroll
        for (int m = 0; m < M2; ++m)
            word_y_p<2, DIAG, MODE>(Ub, M8 + 2 * M4 + 4 * m, sh, X2 + 4 * (slice + 8 * m), cg,
                                    t.alpha * (1.0f / 64.0f), bc, cc, &Y[Y2 + 16 * m]);
    }
    __syncthreads();
    if (tid < 128) {
        if constexpr (PIV) {
            // row-table slot tid holds physical row p, or no row
            int bw;
            const int p = slot_row(t.hi, tid, bw);
            if (p >= 0) {
                refit_row<128, MODE>(sh, tid, p, bw, sh.d.sr[p], rr_out, a.pool.lv);
            } else {
                sh.hrow[tid] = 0.f;
                sh.wrow[tid] = 0.f;
            }
        } else {
            refit_row<128, MODE>(sh, tid, tid, tid < X4 ? 8 : (tid < X2 ? 4 : 2), op.r, rr_out, a.pool.lv);
        }
    }
    __syncthreads();

    // pass 2: yh = y r / r' and the column maxima per width
    {
        float mx8[4] = {0.f, 0.f, 0.f, 0.f}, mx4[4] = {0.f, 0.f, 0.f, 0.f}, mx2[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < M8; ++m) word_scale_max<8>(&Y[4 * m], sh.hrow, slice + 8 * m, mx8);
#pragma unroll
        for (int m = 0; m < M4; ++m) word_scale_max<4>(&Y[Y4 + 8 * m], sh.hrow, X4 + 2 * (slice + 8 * m), mx4);
#pragma unroll
        for (int m = 0; m < M2; ++m) word_scale_max<2>(&Y[Y2 + 16 * m], sh.hrow, X2 + 4 * (slice + 8 * m), mx2);
        sh.u.cmax[slice][cg] = width_max(mx8, mx4, mx2);
    }
    __syncthreads();
    if (tid < 128) refit_colmax<128>(sh, tid);
    __syncthreads();

    // pass 3: fixed codes and the least-squares sums
    {
        float ec[4];
        ld4(&sh.ecol[4 * cg], ec);
        float num[4] = {0.f, 0.f, 0.f, 0.f}, den[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < M8; ++m) word_fit<8>(&Y[4 * m], sh.wrow, slice + 8 * m, ec, num, den);
#pragma unroll
        for (int m = 0; m < M4; ++m) word_fit<4>(&Y[Y4 + 8 * m], sh.wrow, X4 + 2 * (slice + 8 * m), ec, num, den);
#pragma unroll
        for (int m = 0; m < M2; ++m) word_fit<2>(&Y[Y2 + 16 * m], sh.wrow, X2 + 4 * (slice + 8 * m), ec, num, den);
        sh.d.red[0][slice][cg] = make_float4(num[0], num[1], num[2], num[3]);
        sh.d.red[1][slice][cg] = make_float4(den[0], den[1], den[2], den[3]);
    }
    __syncthreads();
    if (tid < 128) refit_colfit<128>(sh, tid, cc_out);
    __syncthreads();

    // pass 4: requantize on the new scales, store in place
    float g[4];
    ld4(&sh.gcol[4 * cg], g);
#pragma unroll
    for (int m = 0; m < M8; ++m) cw.store_m(tid, m, word_requant<8>(&Y[4 * m], g));
#pragma unroll
    for (int m = 0; m < M4; ++m)
        cw.store_m(tid, M8 + m, word_requant<4>(&Y[Y4 + 8 * m], g));
#pragma unroll
    for (int m = 0; m < M2; ++m)
        cw.store_m(tid, M8 + M4 + m, word_requant<2>(&Y[Y2 + 16 * m], g));
}

// ---- any row-width mix and d_v: the words stay packed in registers and
// each pass unpacks them again.

template <int B, bool DIAG, int DV>
__device__ __forceinline__ void gen_word_y(uint32_t w, const DecodeShared<DV> &d, int x0, float alpha,
                                           const float (&bc)[4], float (&Y)[16])
{
    float U[16];
    unpack_word<B>(w, U);
    const float al_w = alpha * (B == 8 ? 1.0f : (B == 4 ? (1.0f / 16.0f) : (1.0f / 64.0f)));
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float a_s = d.av[x0 + s];
        const float al = DIAG ? d.al[x0 + s] : al_w;
#pragma unroll
        for (int e = 0; e < 4; ++e) Y[4 * s + e] = fmaf(al, U[4 * s + e], a_s * bc[e]);
    }
}

// Calls f(width constant, group geometry, word index) for every word of the
// thread that holds codes.
template <int DV, class F>
__device__ __forceinline__ void each_word(const TileCtx &t, int slice, F &&f)
{
    constexpr int NSL = 256 / (DV / 4);
    constexpr int MMAX = kMaxDk * (DV / 4) / 256;
    const int ngroups = static_cast<int>(t.hi.groups);
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
        const int g = slice + NSL * m;
        if (g < ngroups) {
            const GroupRows gr = group_rows(t.hi, g);
            if (gr.bits == 8) f(std::integral_constant<int, 8>(), gr, m);
            else if (gr.bits == 4) f(std::integral_constant<int, 4>(), gr, m);
            else f(std::integral_constant<int, 2>(), gr, m);
        }
    }
}

template <bool BF16, bool DIAG, int DV, Refit MODE>
__device__ __forceinline__ void refit_generic(const DecodeArgs &a, const TileCtx &t, RefitShared<DV> &sh)
{
    constexpr int CG = DV / 4;
    constexpr int NSL = 256 / CG;
    constexpr int MMAX = kMaxDk * CG / 256;
    const int tid = threadIdx.x;
    const int cg = tid % CG, slice = tid / CG;
    const int ngroups = static_cast<int>(t.hi.groups);
    const int dk = a.pool.dk;
    float *rr_out = const_cast<float *>(t.rr);
    float *cc_out = const_cast<float *>(t.cc);
    const CodeWords cw(t.codes, t.hi.piv_off);
    uint32_t w[MMAX];
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
        const int g = slice + NSL * m;
        w[m] = g < ngroups ? cw.load(tid + 256 * m) : 0u;
    }
    PivotRegs<DV> pr;
    pivot_load(t, slice, cg, pr);
    const RowColOps op = load_ops<BF16, DIAG, DV>(a, t.tile, t.b, t.hq, t.h, t.rr, t.cc);
    if (tid < DV) sh.ccol[tid] = op.c;
    if (tid < dk) sh.wphys[tid] = a.pool.roww[t.h * dk + tid];
    const float kappa = row_constants<DIAG, DV>(t.hi, dk, t.alpha, t.beta, op, sh.d, a.pool.lv);

    float acK[4] = {0.f, 0.f, 0.f, 0.f}, acQ[4] = {0.f, 0.f, 0.f, 0.f};
    each_word<DV>(t, slice, [&](auto bw, const GroupRows &gr, int m) {
        float U[16];
        unpack_acc<decltype(bw)::value>(w[m], sh.d.kq, gr.x0, U, acK, acQ);
    });
    pivot_acc(t, slice, cg, pr, sh.d, acK, acQ);
    column_phase<DV>(a, t.tile, DIAG ? 1.0f : t.alpha, t.beta, sh.d, kappa, acK, acQ, op.c, op.v);

    float bc[4], cc[4];
    ld4(&sh.d.bcol[4 * cg], bc);
    ld4(&sh.ccol[4 * cg], cc);
    pivot_update(t, slice, cg, pr, sh.d, bc);      // pivot rows take no part in the fits

    // pass 1: row partials straight to LDS (one entry per lane pair and slot)
    each_word<DV>(t, slice, [&](auto bw, const GroupRows &gr, int m) {
        constexpr int B = decltype(bw)::value;
        float Y[16];
        gen_word_y<B, DIAG, DV>(w[m], sh.d, gr.x0, t.alpha, bc, Y);
#pragma unroll
        for (int s = 0; s < 8 / B; ++s) put_row_partial<DV, MODE>(sh, gr.x0 + s, cg, row_partial<MODE>(&Y[4 * s], cc));
    });
    __syncthreads();
    if (tid < kSlotTable) {
        int bw;
        const int p = slot_row(t.hi, tid, bw);
        if (p >= 0) {
            refit_row<DV, MODE>(sh, tid, p, bw, sh.d.sr[p], rr_out, a.pool.lv);
        } else {
            sh.hrow[tid] = 0.f;
            sh.wrow[tid] = 0.f;
        }
    }
    if constexpr (MODE == Refit::RowAbsmax) {
        if (tid < DV) cc_out[tid] = 1.0f;
    }
    __syncthreads();

    if constexpr (MODE == Refit::RowAbsmax) {
        each_word<DV>(t, slice, [&](auto bw, const GroupRows &gr, int m) {
            constexpr int B = decltype(bw)::value;
            float Y[16];
            gen_word_y<B, DIAG, DV>(w[m], sh.d, gr.x0, t.alpha, bc, Y);
            word_scale<B>(Y, sh.hrow, gr.x0);
            cw.store(tid + 256 * m, word_requant<B>(Y, cc));
        });
        return;
    }

    // pass 2: column maxima of |yh| per width
    {
        float mx[3][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
        each_word<DV>(t, slice, [&](auto bw, const GroupRows &gr, int m) {
            constexpr int B = decltype(bw)::value;
            constexpr int K = B == 8 ? 0 : (B == 4 ? 1 : 2);
            float Y[16];
            gen_word_y<B, DIAG, DV>(w[m], sh.d, gr.x0, t.alpha, bc, Y);
#pragma unroll
            for (int s = 0; s < 8 / B; ++s) {
                const float h = sh.hrow[gr.x0 + s];
#pragma unroll
                for (int e = 0; e < 4; ++e) mx[K][e] = fmaxf(mx[K][e], fabsf(Y[4 * s + e] * h));
            }
        });
        sh.u.cmax[slice][cg] = width_max(mx[0], mx[1], mx[2]);
    }
    __syncthreads();
    if (tid < DV) refit_colmax<DV>(sh, tid);
    __syncthreads();

    // pass 3: fixed codes, least-squares sums
    {
        float ec[4];
        ld4(&sh.ecol[4 * cg], ec);
        float num[4] = {0.f, 0.f, 0.f, 0.f}, den[4] = {0.f, 0.f, 0.f, 0.f};
        each_word<DV>(t, slice, [&](auto bw, const GroupRows &gr, int m) {
            constexpr int B = decltype(bw)::value;
            float Y[16];
            gen_word_y<B, DIAG, DV>(w[m], sh.d, gr.x0, t.alpha, bc, Y);
#pragma unroll
            for (int s = 0; s < 8 / B; ++s) {
                const float h = sh.hrow[gr.x0 + s];
#pragma unroll
                for (int e = 0; e < 4; ++e) Y[4 * s + e] *= h;
            }
            word_fit<B>(Y, sh.wrow, gr.x0, ec, num, den);
        });
        sh.d.red[0][slice][cg] = make_float4(num[0], num[1], num[2], num[3]);
        sh.d.red[1][slice][cg] = make_float4(den[0], den[1], den[2], den[3]);
    }
    __syncthreads();
    if (tid < DV) refit_colfit<DV>(sh, tid, cc_out);
    __syncthreads();

    // pass 4: requantize and store
    float g[4];
    ld4(&sh.gcol[4 * cg], g);
    each_word<DV>(t, slice, [&](auto bw, const GroupRows &gr, int m) {
        constexpr int B = decltype(bw)::value;
        float Y[16];
        gen_word_y<B, DIAG, DV>(w[m], sh.d, gr.x0, t.alpha, bc, Y);
#pragma unroll
        for (int s = 0; s < 8 / B; ++s) {
            const float h = sh.hrow[gr.x0 + s];
#pragma unroll
            for (int e = 0; e < 4; ++e) Y[4 * s + e] *= h;
        }
        cw.store(tid + 256 * m, word_requant<B>(Y, g));
    });
}

// ---- row-mix heads (kRowMix: 8- and 4-bit rows in any split, at most
// kCompactPivots FP16 pivot rows, d = 128: the per-row maps of a row-unit
// calibration).  The first half is the frozen row-mix body's (rowmix_sums:
// both sums over rows on the matrix cores, here all four columns in one
// pass: the register peak comes later).  Then, as in the uniform body, y
// stays in registers through the four passes, indexed by word-step: Y[m]
// holds word-step m's row (an 8-bit word) or the slot-0 row of its 4-bit
// word, at most 64 values; the slot-1 row of a 4-bit word is formed again
// from the packed word in each pass after the first.  The per-element
// arithmetic is the generic body's (gen_word_y, word_fit, word_requant) in
// the same order, so the two bodies give the same codes and scales.
// The width of a word-step is a per-lane test (it differs between slices in
// at most one word-step): measured faster than a uniform branch for the
// word-steps wholly of one width.  Lanes past the head's last group (in the
// last word-step) take no part in the sums and store nothing.

// y of the 4 fields of view W (each at the top of its byte) of row slot x,
// as gen_word_y forms it.
template <bool DIAG>
__device__ __forceinline__ void rm_row_y(uint32_t W, const DecodeShared<128> &d, int x, float al_w,
                                         const float (&bc)[4], float *y)
{
    const float a_s = d.av[x];
    const float al = DIAG ? d.al[x] : al_w;
#pragma unroll
    for (int e = 0; e < 4; ++e) y[e] = fmaf(al, sbyte(W, e), a_s * bc[e]);
}

// Calls f8(m, g) for word-step m of the thread if its group g = slice + 8 m
// is 8-bit, or f4(m, g) if it is a 4-bit group that holds codes (g < ng),
// for every m while 8 m < ng.
template <class F8, class F4>
__device__ __forceinline__ void rm_each_step(int slice, int g8, int ng, F8 &&f8, F4 &&f4)
{
#pragma unroll
    for (int m = 0; m < 16; ++m) {
        if (8 * m >= ng) break;
        const int g = slice + 8 * m;
        if (g < g8) f8(m, g);
        else if (g < ng) f4(m, g);
    }
}

template <bool BF16, bool DIAG>
__device__ __forceinline__ void refit_rowmix(const DecodeArgs &a, const TileCtx &t, RefitShared<128> &sh)
{
    constexpr Refit DA = Refit::DualAxis;
    const int tid = threadIdx.x;
    const int cg = tid & 31, slice = tid >> 5;
    const int g8 = __builtin_amdgcn_readfirstlane(static_cast<int>(t.hi.g8));
    const int ng = __builtin_amdgcn_readfirstlane(static_cast<int>(t.hi.groups));
    float *rr_out = const_cast<float *>(t.rr);
    float *cc_out = const_cast<float *>(t.cc);
    // the buffer covers the codes region only (piv_off = 128 ng): words of
    // groups past the head's last read 0
    const CodeWords cw(t.codes, t.hi.piv_off);
    uint32_t w[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) w[m] = 8 * m < ng ? cw.load(tid + 256 * m) : 0u;
    PivotRegs<128, kCompactPivots> pr;
    pivot_load<128, kCompactPivots>(t, slice, cg, pr);
    const RowColOps op = load_ops<BF16, DIAG, 128>(a, t.tile, t.b, t.hq, t.h, t.rr, t.cc);
    if (tid < 128) {
        sh.ccol[tid] = op.c;
        sh.wphys[tid] = a.pool.roww[t.h * 128 + tid];
    }
    rowmix_sums<DIAG, false, true>(a, t, sh.d, w, pr, op, g8, ng);

    float bc[4], cc[4];
    ld4(&sh.d.bcol[4 * cg], bc);
    ld4(&sh.ccol[4 * cg], cc);
    pivot_update<128, kCompactPivots>(t, slice, cg, pr, sh.d, bc);    // pivot rows take no part in the fits
    const float al8 = t.alpha, al4 = t.alpha * (1.0f / 16.0f);

    // pass 1: y on the old scales, the row partials (row slot g of an 8-bit
    // group, 2 g - g8 and the next of a 4-bit one)
    float Y[16][4];
    rm_each_step(
        slice, g8, ng,
        [&](int m, int g) {
            rm_row_y<DIAG>(w[m], sh.d, g, al8, bc, Y[m]);
            put_row_partial<128, DA>(sh, g, cg, row_partial<DA>(Y[m], cc));
        },
        [&](int m, int g) {
            const int x0 = 2 * g - g8;
            float y1[4];
            rm_row_y<DIAG>(slot_top<4>(w[m], 0), sh.d, x0, al4, bc, Y[m]);
            rm_row_y<DIAG>(slot_top<4>(w[m], 1), sh.d, x0 + 1, al4, bc, y1);
            put_row_partial<128, DA>(sh, x0, cg, row_partial<DA>(Y[m], cc));
            put_row_partial<128, DA>(sh, x0 + 1, cg, row_partial<DA>(y1, cc));
        });
    __syncthreads();
    if (tid < kSlotTable) {
        int bw;
        const int p = slot_row(t.hi, tid, bw);
        if (p >= 0) {
            refit_row<128, DA>(sh, tid, p, bw, sh.d.sr[p], rr_out, a.pool.lv);
        } else {
            sh.hrow[tid] = 0.f;
            sh.wrow[tid] = 0.f;
        }
    }
    __syncthreads();

    // yh of the slot-1 row of the 4-bit word of word-step m, group g
    auto slot1_yh = [&](int m, int g, float (&y1)[4]) {
        const int x1 = 2 * g - g8 + 1;
        rm_row_y<DIAG>(slot_top<4>(w[m], 1), sh.d, x1, al4, bc, y1);
        const float h = sh.hrow[x1];
#pragma unroll
        for (int e = 0; e < 4; ++e) y1[e] *= h;
    };

    // pass 2: yh = y r / r' (in place for the kept rows) and the column
    // maxima per width
    {
        float mx8[4] = {0.f, 0.f, 0.f, 0.f}, mx4[4] = {0.f, 0.f, 0.f, 0.f};
        const float mx2[4] = {0.f, 0.f, 0.f, 0.f};
        rm_each_step(
            slice, g8, ng,
            [&](int m, int g) {
                const float h = sh.hrow[g];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    Y[m][e] *= h;
                    mx8[e] = fmaxf(mx8[e], fabsf(Y[m][e]));
                }
            },
            [&](int m, int g) {
                const float h = sh.hrow[2 * g - g8];
                float y1[4];
                slot1_yh(m, g, y1);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    Y[m][e] *= h;
                    mx4[e] = fmaxf(mx4[e], fabsf(Y[m][e]));
                    mx4[e] = fmaxf(mx4[e], fabsf(y1[e]));
                }
            });
        sh.u.cmax[slice][cg] = width_max(mx8, mx4, mx2);
    }
    __syncthreads();
    if (tid < 128) refit_colmax<128>(sh, tid);
    __syncthreads();

    // pass 3: fixed codes and the least-squares sums
    {
        float ec[4];
        ld4(&sh.ecol[4 * cg], ec);
        float num[4] = {0.f, 0.f, 0.f, 0.f}, den[4] = {0.f, 0.f, 0.f, 0.f};
        rm_each_step(
            slice, g8, ng, [&](int m, int g) { word_fit<8>(Y[m], sh.wrow, g, ec, num, den); },
            [&](int m, int g) {
                float y8[8];
                slot1_yh(m, g, *reinterpret_cast<float(*)[4]>(&y8[4]));
#pragma unroll
                for (int e = 0; e < 4; ++e) y8[e] = Y[m][e];
                word_fit<4>(y8, sh.wrow, 2 * g - g8, ec, num, den);
            });
        sh.d.red[0][slice][cg] = make_float4(num[0], num[1], num[2], num[3]);
        sh.d.red[1][slice][cg] = make_float4(den[0], den[1], den[2], den[3]);
    }
    __syncthreads();
    if (tid < 128) refit_colfit<128>(sh, tid, cc_out);
    __syncthreads();

    // pass 4: requantize on the new scales, store in place
    float gc[4];
    ld4(&sh.gcol[4 * cg], gc);
    rm_each_step(
        slice, g8, ng, [&](int m, int) { cw.store(tid + 256 * m, word_requant<8>(Y[m], gc)); },
        [&](int m, int g) {
            float y8[8];
            slot1_yh(m, g, *reinterpret_cast<float(*)[4]>(&y8[4]));
#pragma unroll
            for (int e = 0; e < 4; ++e) y8[e] = Y[m][e];
            cw.store(tid + 256 * m, word_requant<4>(y8, gc));
        });
}

// A tile of uniform layout L: codes (1024 bytes per word-step), then r, c.
template <bool BF16, bool DIAG, int L, Refit MODE>
__device__ __forceinline__ void run_refit_uniform(const DecodeArgs &a, TileCtx &t, int slot, RefitShared<128> &sh)
{
    constexpr UniformLayout u = kUniformLayouts[L - 1];
    constexpr uint32_t r_off = 1024u * (u.m8 + u.m4 + u.m2);
    uint8_t *rec = a.pool.base + static_cast<uint64_t>(slot) * a.pool.slot_bytes + t.off;
    t.codes = reinterpret_cast<uint32_t *>(rec);
    t.rr = reinterpret_cast<const float *>(rec + r_off);
    t.cc = t.rr + 128;
    refit_uniform<BF16, DIAG, u.m8, u.m4, u.m2, MODE>(a, t, sh);
}

// A padded pivot head of uniform layout L (its row counts from the head
// list), or a layout-L head taken as one with no pivot rows.
template <bool BF16, bool DIAG, int L, Refit MODE>
__device__ __forceinline__ void run_refit_uniform_piv(const DecodeArgs &a, TileCtx &t, int slot, RefitShared<128> &sh)
{
    constexpr UniformLayout u = kUniformLayouts[L - 1];
    padded_pivot_tile<L>(a, t, slot);
    refit_uniform<BF16, DIAG, u.m8, u.m4, u.m2, MODE, true>(a, t, sh);
}

template <int DV, bool BF16, int LAYOUT, bool DIAG, Refit MODE>
__global__ __launch_bounds__(256) void refit_kernel(DecodeArgs a)
{
    __shared__ RefitShared<DV> sh;
    const PoolView &P = a.pool;
    TileCtx t;
    uint32_t tile_bytes = 0;
    constexpr bool UNIFORM = DV == 128 && LAYOUT > 0 && LAYOUT <= kNumUniformLayouts;
    if constexpr (UNIFORM) {
        constexpr UniformLayout u = kUniformLayouts[LAYOUT - 1];
        tile_bytes = 1024u * (u.m8 + u.m4 + u.m2 + 1);
    }
    tile_of(a, tile_bytes, t);
    const int slot = a.slot_ids[t.b];
    t.alpha = DIAG ? 1.0f : act_ld<BF16>(a.alpha, t.tile);
    t.beta = act_ld<BF16>(a.beta, t.tile);
    if constexpr (UNIFORM) {
        run_refit_uniform<BF16, DIAG, LAYOUT, MODE>(a, t, slot, sh);
    } else if constexpr (DV == 128 && LAYOUT > kPivotUniformBase && LAYOUT <= kPivotUniformBase + kNumUniformLayouts) {
        run_refit_uniform_piv<BF16, DIAG, LAYOUT - kPivotUniformBase, MODE>(a, t, slot, sh);
    } else if constexpr (DV == 128 && LAYOUT > kMixedPivotBase && LAYOUT <= kMixedPivotBase + 2) {
        // layout-L heads and layout-L padded pivot heads in one launch of one
        // body: a layout-L head is a padded pivot head with no pivot rows
        run_refit_uniform_piv<BF16, DIAG, LAYOUT - kMixedPivotBase, MODE>(a, t, slot, sh);
    } else if constexpr (DV == 128 && LAYOUT == kMultiUniform) {
        // heads of several uniform layouts and whole FP16 heads in one launch
        // (the head list), each tile on its own body; a whole FP16 head has
        // no integer rows to fit and takes the frozen-step body
        switch (t.layout) {
        case 1: run_refit_uniform<BF16, DIAG, 1, MODE>(a, t, slot, sh); break;
        case 2: run_refit_uniform<BF16, DIAG, 2, MODE>(a, t, slot, sh); break;
        case 3: run_refit_uniform<BF16, DIAG, 3, MODE>(a, t, slot, sh); break;
        case 4: run_refit_uniform<BF16, DIAG, 4, MODE>(a, t, slot, sh); break;
        case 5: run_refit_uniform<BF16, DIAG, 5, MODE>(a, t, slot, sh); break;
        default: run_f16head<BF16, DIAG>(a, t, slot, sh.d); break;
        }
    } else {
        t.hi = P.heads[t.h];
        uint8_t *rec = P.base + static_cast<uint64_t>(slot) * P.slot_bytes + t.hi.tile_off;
        t.codes = reinterpret_cast<uint32_t *>(rec);
        t.rr = reinterpret_cast<const float *>(rec + t.hi.r_off);
        t.cc = t.rr + P.dk;
        if constexpr (DV == 128 && LAYOUT == kRowMix) {
            static_assert(MODE == Refit::DualAxis, "the row-mix refitting body runs the dual-axis fit");
            refit_rowmix<BF16, DIAG>(a, t, sh);
        } else {
            refit_generic<BF16, DIAG, DV, MODE>(a, t, sh);
        }
    }
}

template <bool BF16, bool DIAG, Refit MODE>
hipError_t launch_refit_any(const DecodeArgs &a, int layout, unsigned grid, hipStream_t s)
{
    if constexpr (MODE == Refit::RowAbsmax) {
        // uniform layouts are launched on the lean body (launch_decode_rowmax)
        if (a.pool.dv == 128) hipLaunchKernelGGL((refit_kernel<128, BF16, 0, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
        else hipLaunchKernelGGL((refit_kernel<64, BF16, 0, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
    } else if (a.pool.dv == 128) {
        switch (layout) {
        case 1: hipLaunchKernelGGL((refit_kernel<128, BF16, 1, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a); break;
        case 2: hipLaunchKernelGGL((refit_kernel<128, BF16, 2, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a); break;
        case 3: hipLaunchKernelGGL((refit_kernel<128, BF16, 3, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a); break;
        case 4: hipLaunchKernelGGL((refit_kernel<128, BF16, 4, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a); break;
        case 5: hipLaunchKernelGGL((refit_kernel<128, BF16, 5, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a); break;
        case kRowMix:
            hipLaunchKernelGGL((refit_kernel<128, BF16, kRowMix, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
            break;
        case kMultiUniform:
            hipLaunchKernelGGL((refit_kernel<128, BF16, kMultiUniform, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
            break;
        case kPivotUniformBase + 1:
            hipLaunchKernelGGL((refit_kernel<128, BF16, kPivotUniformBase + 1, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
            break;
        case kPivotUniformBase + 2:
            hipLaunchKernelGGL((refit_kernel<128, BF16, kPivotUniformBase + 2, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
            break;
        case kPivotUniformBase + 3:
            hipLaunchKernelGGL((refit_kernel<128, BF16, kPivotUniformBase + 3, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
            break;
        case kPivotUniformBase + 4:
            hipLaunchKernelGGL((refit_kernel<128, BF16, kPivotUniformBase + 4, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
            break;
        case kPivotUniformBase + 5:
            hipLaunchKernelGGL((refit_kernel<128, BF16, kPivotUniformBase + 5, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
            break;
        case kMixedPivotBase + 1:
            hipLaunchKernelGGL((refit_kernel<128, BF16, kMixedPivotBase + 1, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
            break;
        case kMixedPivotBase + 2:
            hipLaunchKernelGGL((refit_kernel<128, BF16, kMixedPivotBase + 2, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
            break;
        default: hipLaunchKernelGGL((refit_kernel<128, BF16, 0, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a); break;
        }
    } else {
        hipLaunchKernelGGL((refit_kernel<64, BF16, 0, DIAG, MODE>), dim3(grid), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

template <Refit MODE>
hipError_t launch_refit_mode(const DecodeArgs &a, bool bf16, bool diag, int pool_layout, hipStream_t stream)
{
    const unsigned grid = static_cast<unsigned>(a.batch) * static_cast<unsigned>(a.n_heads);
    if (grid == 0) return hipSuccess;
    if (bf16) return diag ? launch_refit_any<true, true, MODE>(a, pool_layout, grid, stream)
                          : launch_refit_any<true, false, MODE>(a, pool_layout, grid, stream);
    return diag ? launch_refit_any<false, true, MODE>(a, pool_layout, grid, stream)
                : launch_refit_any<false, false, MODE>(a, pool_layout, grid, stream);
}

}  // namespace
}  // namespace stepq
