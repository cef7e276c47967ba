// Kernels of libstepq for gfx950 (CDNA4, wave64).
//
// decode_kernel: the fused quantized gated-Delta decode step, one 256-thread
// workgroup per (request, value head) tile.  The math is arranged in "code
// space" so that the tile is never materialised in floating point:
//
//   with U_ij = 2^(8-b_i) q_ij (what a sign-extending byte read of a b-bit
//   field left-aligned in its byte yields) and f_i = 2^(b_i-8):
//     (S^T k)_j = c_j sum_i [k_i r_i f_i / q_b]  U_ij          (Section 4.3 reconstruction)
//     (S^T q)_j = c_j sum_i [q_i r_i f_i / q_b]  U_ij
//     delta_j   = v_j - alpha (S^T k)_j                         (Eq. 1 residual)
//     o_j       = alpha (S^T q)_j + beta (q^T k) delta_j        (= X^T q, Eq. 4)
//     X_ij q_b/(r_i c_j) = (alpha f_i) U_ij + [beta k_i q_b / r_i] [delta_j / c_j]
//   so the requantized code (Eq. 3) is round-to-even of a rank-1 update of
//   the old code, clamped to +-q_b.
//
// Work split: the tile's codes region is a run of 32-bit words; thread t owns
// words t + 256 m.  At d_v = 128 a row group is 32 words, so a thread always
// owns the same 4 columns (word t % 32) in groups t/32 + 8 m, and a
// wavefront's load covers two whole 128-byte groups.  Per-column partial sums
// of the 8 threads that share a column meet in LDS; one pass over the words
// kept in registers then rewrites the codes in place.
//
// tile_kernel: pack (from fp32 states or raw codes), unpack and dequantize
// whole tiles; not on the decode path.
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

__device__ __forceinline__ GroupRows group_rows(const HeadInfo &hi, int g)
{
    if (g < hi.g8) return {8, 1, g, hi.n8, g};
    if (g < hi.g8 + hi.g4) {
        const int k = g - hi.g8;
        return {4, 2, hi.n8 + 2 * k, hi.n8 + hi.n4, hi.n8 + 2 * k};
    }
    const int k = g - hi.g8 - hi.g4;
    return {2, 4, hi.n8 + hi.n4 + 4 * k, hi.n8 + hi.n4 + hi.n2, hi.n8 + 2 * hi.g4 + 4 * k};
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
};

struct TileCtx {
    int tile, b, h, hq;
    HeadInfo hi;
    uint32_t *codes;
    const float *rr, *cc;
    float alpha, beta;
};

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
template <bool DIAG, int DV>
__device__ __forceinline__ float row_constants(const HeadInfo &hi, int dk, float beta, const RowColOps &op,
                                               DecodeShared<DV> &sh)
{
    const int tid = threadIdx.x;
    if (tid < dk) {
        sh.sk[tid] = op.k;
        sh.sq[tid] = op.q;
        sh.sr[tid] = op.r;
        sh.sperm[tid] = op.perm;
        if constexpr (DIAG) sh.sd[tid] = op.d;
    }
    __syncthreads();
    float kq = 0.f;
    if (tid < kSlotTable) {
        const int x = tid;
        int bw = 8, p = -1;
        if (x < hi.n8) {
            p = x;
        } else if (x < hi.n8 + 2 * hi.g4) {
            bw = 4;
            const int kk = x - hi.n8;
            if (kk < hi.n4) p = hi.n8 + kk;
        } else if (x < hi.n8 + 2 * hi.g4 + 4 * hi.g2) {
            bw = 2;
            const int kk = x - hi.n8 - 2 * hi.g4;
            if (kk < hi.n2) p = hi.n8 + hi.n4 + kk;
        }
        float kt = 0.f, qt = 0.f, av = 0.f, al = 0.f;
        if (p >= 0) {
            // slot x holds physical row p, whose r and permutation entry were
            // loaded by thread p
            const int i = sh.sperm[p];
            const float ki = sh.sk[i];
            const float qi = sh.sq[i];
            const float rp = sh.sr[p];
            const float qb = bw == 8 ? 127.0f : (bw == 4 ? 7.0f : 1.0f);
            // 2^(b-8) / q_b: 1/127, 1/112, 1/64 (an unpacked field reads 2^(8-b) q)
            const float fq = bw == 8 ? (1.0f / 127.0f) : (bw == 4 ? (1.0f / 112.0f) : (1.0f / 64.0f));
            const float di = DIAG ? sh.sd[i] : 1.0f;       // the gate folds into both row weights
            const float rs = rp * fq * di;
            kt = ki * rs;
            qt = qi * rs;
            av = beta * ki * qb * __builtin_amdgcn_rcpf(rp);
            al = di * (bw == 8 ? 1.0f : (bw == 4 ? (1.0f / 16.0f) : (1.0f / 64.0f)));
            kq = qi * ki;
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

// Uniform layouts: table slot = physical row = tid, widths known at compile time.
template <bool DIAG, int M8, int M4, int DV>
__device__ __forceinline__ float row_constants_uniform(float beta, const RowColOps &op, DecodeShared<DV> &sh)
{
    constexpr int X4 = 8 * M8, X2 = 8 * M8 + 16 * M4;
    const int tid = threadIdx.x;
    if (tid < 128) {
        sh.sk[tid] = op.k;
        sh.sq[tid] = op.q;
        if constexpr (DIAG) sh.sd[tid] = op.d;
    }
    __syncthreads();
    float kq = 0.f;
    if (tid < 128) {
        const int p = tid;
        const float qb = p < X4 ? 127.0f : (p < X2 ? 7.0f : 1.0f);
        const float fq = p < X4 ? (1.0f / 127.0f) : (p < X2 ? (1.0f / 112.0f) : (1.0f / 64.0f));
        const float ki = sh.sk[op.perm];
        const float qi = sh.sq[op.perm];
        const float di = DIAG ? sh.sd[op.perm] : 1.0f;
        const float rs = op.r * fq * di;
        sh.kq[p] = make_float2(ki * rs, qi * rs);
        sh.av[p] = beta * ki * qb * __builtin_amdgcn_rcpf(op.r);
        if constexpr (DIAG) sh.al[p] = di * (p < X4 ? 1.0f : (p < X2 ? (1.0f / 16.0f) : (1.0f / 64.0f)));
        kq = qi * ki;
    }
    kq = wave_sum(kq);
    if ((tid & 63) == 0) sh.kap[tid >> 6] = kq;
    __syncthreads();
    return (sh.kap[0] + sh.kap[1]) + (sh.kap[2] + sh.kap[3]);
}

// Column sums of the per-thread partials, residual, readout, column factor
// of the code-space update.  cj, vj: column tid's scale and value (threads
// < DV, loaded at the start of the tile).  Ends with a barrier.
template <int DV>
__device__ __forceinline__ void column_phase(const DecodeArgs &a, int tile, float alpha, float beta,
                                             DecodeShared<DV> &sh, float kappa, const float (&acK)[4],
                                             const float (&acQ)[4], float cj, float vj)
{
    constexpr int CG = DV / 4, NSL = 256 / CG;
    const int tid = threadIdx.x;
    sh.red[0][tid / CG][tid % CG] = make_float4(acK[0], acK[1], acK[2], acK[3]);
    sh.red[1][tid / CG][tid % CG] = make_float4(acQ[0], acQ[1], acQ[2], acQ[3]);
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

// ---- codes kept as packed f16 pairs between the passes (exact: |2^(8-B) q| <= 127)

// Bytes LO and HI of w, read as signed, to an f16 pair: one SDWA convert per
// field, the second one writing the upper half in place.
template <int LO, int HI>
__device__ __forceinline__ uint32_t sbytes_f16(uint32_t w)
{
    uint32_t r;
    asm("v_cvt_f16_i16_sdwa %0, sext(%1) dst_sel:WORD_0 dst_unused:UNUSED_PAD src0_sel:BYTE_%c2"
        : "=v"(r) : "v"(w), "i"(LO));
    asm("v_cvt_f16_i16_sdwa %0, sext(%1) dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:BYTE_%c2"
        : "+v"(r) : "v"(w), "i"(HI));
    return r;
}

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

template <int E>
__device__ __forceinline__ float fma_mix_e(float a, const uint32_t *U2, int s, float c)
{
    return fma_mix<E & 1>(a, U2[2 * s + (E >> 1)], c);
}

template <int B>
__device__ __forceinline__ void unpack_acc_h(uint32_t w, const float2 *kq, int x0, uint32_t *U2, float (&acK)[4],
                                             float (&acQ)[4])
{
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float2 c = kq[x0 + s];
        const uint32_t W = slot_top<B>(w, s);
        U2[2 * s] = sbytes_f16<0, 1>(W);
        U2[2 * s + 1] = sbytes_f16<2, 3>(W);
        acK[0] = fma_mix_e<0>(c.x, U2, s, acK[0]);
        acQ[0] = fma_mix_e<0>(c.y, U2, s, acQ[0]);
        acK[1] = fma_mix_e<1>(c.x, U2, s, acK[1]);
        acQ[1] = fma_mix_e<1>(c.y, U2, s, acQ[1]);
        acK[2] = fma_mix_e<2>(c.x, U2, s, acK[2]);
        acQ[2] = fma_mix_e<2>(c.y, U2, s, acQ[2]);
        acK[3] = fma_mix_e<3>(c.x, U2, s, acK[3]);
        acQ[3] = fma_mix_e<3>(c.y, U2, s, acQ[3]);
    }
}

template <int B, int E>
__device__ __forceinline__ uint32_t requant_field(const uint32_t *U2, int s, float al, float a_s, float bce, uint32_t P)
{
    constexpr float bias = static_cast<float>(1 << (B - 1));
    constexpr float top = static_cast<float>((1 << B) - 1);
    const float tt = fmaf(a_s, bce, bias);
    float y = fma_mix_e<E>(al, U2, s, tt);
    y = __builtin_amdgcn_fmed3f(y, 1.0f, top);
    return __builtin_amdgcn_cvt_pk_u8_f32(y, E, P);
}

// al: the per-width gate factor (scalar gate) or, with a table alt, per row.
template <int B, bool DIAG>
__device__ __forceinline__ uint32_t requant_word_h(const uint32_t *U2, const float *av, const float *alt, int x0,
                                                   float al_w, const float (&bc)[4])
{
    constexpr uint32_t flip = B == 8 ? 0x80808080u : (B == 4 ? 0x88888888u : 0xAAAAAAAAu);
    uint32_t out = 0;
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float a_s = av[x0 + s];
        const float al = DIAG ? alt[x0 + s] : al_w;
        uint32_t P = 0;
        P = requant_field<B, 0>(U2, s, al, a_s, bc[0], P);
        P = requant_field<B, 1>(U2, s, al, a_s, bc[1], P);
        P = requant_field<B, 2>(U2, s, al, a_s, bc[2], P);
        P = requant_field<B, 3>(U2, s, al, a_s, bc[3], P);
        out |= P << (s * B);
    }
    return out ^ flip;
}

// New word from the unpacked old fields: per field
//   y = al U + av_i bc_j + 2^(B-1)        (code + bias, Eq. 3 argument)
// clamped to [1, 2^B - 1] (i.e. code in [-q_b, q_b]), rounded to nearest
// even and packed to a byte by v_cvt_pk_u8_f32, then the bias is removed
// from all fields at once by flipping each field's top bit.
template <int B, bool DIAG>
__device__ __forceinline__ uint32_t requant_word(const float *U, const float *av, const float *alt, int x0,
                                                 float al_w, const float (&bc)[4])
{
    constexpr float bias = static_cast<float>(1 << (B - 1));
    constexpr float top = static_cast<float>((1 << B) - 1);
    constexpr uint32_t flip = B == 8 ? 0x80808080u : (B == 4 ? 0x88888888u : 0xAAAAAAAAu);
    uint32_t out = 0;
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float a_s = av[x0 + s];
        const float al = DIAG ? alt[x0 + s] : al_w;
        uint32_t P = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float tt = fmaf(a_s, bc[e], bias);
            float y = fmaf(al, U[4 * s + e], tt);
            y = __builtin_amdgcn_fmed3f(y, 1.0f, top);
            P = __builtin_amdgcn_cvt_pk_u8_f32(y, e, P);
        }
        out |= P << (s * B);
    }
    return out ^ flip;
}

// Rows of one width per word-step; codes stay in registers between passes.
template <bool BF16, bool DIAG, int M8, int M4, int M2>
__device__ __forceinline__ void decode_uniform(const DecodeArgs &a, const TileCtx &t, DecodeShared<128> &sh)
{
    constexpr int M = M8 + M4 + M2;
    constexpr int NE = 4 * (M8 + 2 * M4 + 4 * M2);
    constexpr int X4 = 8 * M8, X2 = 8 * M8 + 16 * M4;    // row-table starts of the 4- and 2-bit slots
    const int tid = threadIdx.x;
    const int cg = tid & 31, slice = tid >> 5;
    uint32_t w[M];
#pragma unroll
    for (int m = 0; m < M; ++m) w[m] = __builtin_nontemporal_load(t.codes + tid + 256 * m);

    const RowColOps op = load_ops<BF16, DIAG, 128>(a, t.tile, t.b, t.hq, t.h, t.rr, t.cc);
    const float kappa = row_constants_uniform<DIAG, M8, M4, 128>(t.beta, op, sh);

    uint32_t U[NE / 2];
    float acK[4] = {0.f, 0.f, 0.f, 0.f}, acQ[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int m = 0; m < M8; ++m) unpack_acc_h<8>(w[m], sh.kq, slice + 8 * m, &U[2 * m], acK, acQ);
#pragma unroll
    for (int m = 0; m < M4; ++m)
        unpack_acc_h<4>(w[M8 + m], sh.kq, X4 + 2 * (slice + 8 * m), &U[2 * M8 + 4 * m], acK, acQ);
#pragma unroll
    for (int m = 0; m < M2; ++m)
        unpack_acc_h<2>(w[M8 + M4 + m], sh.kq, X2 + 4 * (slice + 8 * m), &U[2 * M8 + 4 * M4 + 8 * m], acK, acQ);

    column_phase<128>(a, t.tile, DIAG ? 1.0f : t.alpha, t.beta, sh, kappa, acK, acQ, op.c, op.v);

    const float4 b4 = *reinterpret_cast<const float4 *>(&sh.bcol[4 * cg]);
    const float bc[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
    for (int m = 0; m < M8; ++m)
        __builtin_nontemporal_store(requant_word_h<8, DIAG>(&U[2 * m], sh.av, sh.al, slice + 8 * m, t.alpha, bc),
                                    t.codes + tid + 256 * m);
#pragma unroll
    for (int m = 0; m < M4; ++m)
        __builtin_nontemporal_store(requant_word_h<4, DIAG>(&U[2 * M8 + 4 * m], sh.av, sh.al, X4 + 2 * (slice + 8 * m),
                                                    t.alpha * (1.0f / 16.0f), bc),
                                    t.codes + tid + 256 * (M8 + m));
#pragma unroll
    for (int m = 0; m < M2; ++m)
        __builtin_nontemporal_store(requant_word_h<2, DIAG>(&U[2 * M8 + 4 * M4 + 8 * m], sh.av, sh.al, X2 + 4 * (slice + 8 * m),
                                                    t.alpha * (1.0f / 64.0f), bc),
                                    t.codes + tid + 256 * (M8 + M4 + m));
}

// Any row-width mix and d_v: the class of each word-step is looked up at run
// time and the words are unpacked again for the second pass.
template <bool BF16, bool DIAG, int DV>
__device__ __forceinline__ void decode_generic(const DecodeArgs &a, const TileCtx &t, DecodeShared<DV> &sh)
{
    constexpr int CG = DV / 4;
    constexpr int NSL = 256 / CG;
    constexpr int MMAX = kMaxDk * CG / 256;
    const int tid = threadIdx.x;
    const int cg = tid % CG, slice = tid / CG;
    const int ngroups = static_cast<int>(t.hi.groups);
    uint32_t w[MMAX];
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
        const int g = slice + NSL * m;
        w[m] = g < ngroups ? __builtin_nontemporal_load(t.codes + tid + 256 * m) : 0u;
    }
    const RowColOps op = load_ops<BF16, DIAG, DV>(a, t.tile, t.b, t.hq, t.h, t.rr, t.cc);
    const float kappa = row_constants<DIAG, DV>(t.hi, a.pool.dk, t.beta, op, sh);

    float acK[4] = {0.f, 0.f, 0.f, 0.f}, acQ[4] = {0.f, 0.f, 0.f, 0.f};
    float U[16];
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
        const int g = slice + NSL * m;
        if (g < ngroups) {
            const GroupRows gr = group_rows(t.hi, g);
            if (gr.bits == 8) unpack_acc<8>(w[m], sh.kq, gr.x0, U, acK, acQ);
            else if (gr.bits == 4) unpack_acc<4>(w[m], sh.kq, gr.x0, U, acK, acQ);
            else unpack_acc<2>(w[m], sh.kq, gr.x0, U, acK, acQ);
        }
    }
    column_phase<DV>(a, t.tile, DIAG ? 1.0f : t.alpha, t.beta, sh, kappa, acK, acQ, op.c, op.v);

    const float4 b4 = *reinterpret_cast<const float4 *>(&sh.bcol[4 * cg]);
    const float bc[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
        const int g = slice + NSL * m;
        if (g < ngroups) {
            const GroupRows gr = group_rows(t.hi, g);
            uint32_t nw;
            if (gr.bits == 8) {
                unpack_word<8>(w[m], U);
                nw = requant_word<8, DIAG>(U, sh.av, sh.al, gr.x0, t.alpha, bc);
            } else if (gr.bits == 4) {
                unpack_word<4>(w[m], U);
                nw = requant_word<4, DIAG>(U, sh.av, sh.al, gr.x0, t.alpha * (1.0f / 16.0f), bc);
            } else {
                unpack_word<2>(w[m], U);
                nw = requant_word<2, DIAG>(U, sh.av, sh.al, gr.x0, t.alpha * (1.0f / 64.0f), bc);
            }
            __builtin_nontemporal_store(nw, t.codes + tid + 256 * m);
        }
    }
}

// LAYOUT > 0: every head of the pool has uniform layout LAYOUT (checked on
// the host), so the kernel holds only that body and its register budget.
// LAYOUT == 0: heads may differ; each workgroup branches on its head's
// layout (uniformly, so without divergence); d_v = 64 and irregular
// row-width mixes take the generic body.
template <int DV, bool BF16, int LAYOUT, bool DIAG>
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a)
{
    __shared__ DecodeShared<DV> sh;
    const PoolView &P = a.pool;
    TileCtx t;
    t.tile = xcd_tile(blockIdx.x, a.batch * P.Hv);
    t.b = fdiv(t.tile, P.div_hv);
    t.h = t.tile - t.b * P.Hv;
    t.hq = fdiv(t.h, P.div_g);
    const int slot = a.slot_ids[t.b];
    t.alpha = DIAG ? 1.0f : act_ld<BF16>(a.alpha, t.tile);
    t.beta = act_ld<BF16>(a.beta, t.tile);
    if constexpr (DV == 128 && LAYOUT > 0) {
        // every tile record is (codes: 1024 bytes per word-step) + r + c
        constexpr UniformLayout u = kUniformLayouts[LAYOUT - 1];
        constexpr uint32_t r_off = 1024u * (u.m8 + u.m4 + u.m2);
        uint8_t *rec = P.base + static_cast<uint64_t>(slot) * P.slot_bytes +
                       static_cast<uint64_t>(t.h) * (r_off + 1024u);
        t.codes = reinterpret_cast<uint32_t *>(rec);
        t.rr = reinterpret_cast<const float *>(rec + r_off);
        t.cc = t.rr + 128;
        decode_uniform<BF16, DIAG, u.m8, u.m4, u.m2>(a, t, sh);
    } else {
        t.hi = P.heads[t.h];
        uint8_t *rec = P.base + static_cast<uint64_t>(slot) * P.slot_bytes + t.hi.tile_off;
        t.codes = reinterpret_cast<uint32_t *>(rec);
        t.rr = reinterpret_cast<const float *>(rec + t.hi.r_off);
        t.cc = t.rr + P.dk;
        if constexpr (DV == 128) {
            switch (t.hi.layout) {
            case 1: decode_uniform<BF16, DIAG, 8, 4, 0>(a, t, sh); return;
            case 2: decode_uniform<BF16, DIAG, 4, 2, 2>(a, t, sh); return;
            case 3: decode_uniform<BF16, DIAG, 16, 0, 0>(a, t, sh); return;
            case 4: decode_uniform<BF16, DIAG, 0, 8, 0>(a, t, sh); return;
            case 5: decode_uniform<BF16, DIAG, 0, 0, 4>(a, t, sh); return;
            default: break;
            }
        }
        decode_generic<BF16, DIAG, DV>(a, t, sh);
    }
}

// ---------------------------------------------------------------------------
template <TileOp OP>
__global__ __launch_bounds__(256) void tile_kernel(TileArgs a)
{
    const PoolView &P = a.pool;
    const int tid = threadIdx.x;
    const int tile = blockIdx.x;
    const int n_i = tile / P.Hv;
    const int h = tile - n_i * P.Hv;
    const HeadInfo hi = P.heads[h];
    const int slot = a.slot_ids[n_i];
    uint8_t *rec = P.base + static_cast<uint64_t>(slot) * P.slot_bytes + hi.tile_off;
    uint32_t *codes = reinterpret_cast<uint32_t *>(rec);
    float *rr = reinterpret_cast<float *>(rec + hi.r_off);
    float *cc = rr + P.dk;
    const uint8_t *perm = P.perm + h * P.dk;
    const int dk = P.dk, dv = P.dv, CG = dv / 4;
    const size_t tdk = static_cast<size_t>(tile) * dk, tdv = static_cast<size_t>(tile) * dv;

    if constexpr (OP == TileOp::Load || OP == TileOp::Import) {
        for (int p = tid; p < dk; p += 256) rr[p] = a.r_in[tdk + perm[p]];
        for (int j = tid; j < dv; j += 256) cc[j] = a.c_in[tdv + j];
        // zero padding: end of the codes region and end of the record
        uint32_t *rec32 = reinterpret_cast<uint32_t *>(rec);
        for (uint32_t d = hi.groups * CG + tid; d < hi.r_off / 4; d += 256) rec32[d] = 0u;
        for (uint32_t d = (hi.r_off + 4u * (dk + dv)) / 4 + tid; d < hi.tile_bytes / 4; d += 256) rec32[d] = 0u;
    }
    if constexpr (OP == TileOp::Export) {
        for (int p = tid; p < dk; p += 256) a.r_out[tdk + perm[p]] = rr[p];
        for (int j = tid; j < dv; j += 256) a.c_out[tdv + j] = cc[j];
    }

    const int nw = static_cast<int>(hi.groups) * CG;
    for (int d = tid; d < nw; d += 256) {
        const int g = d / CG;
        const int j0 = 4 * (d - g * CG);
        const GroupRows gr = group_rows(hi, g);
        const int B = gr.bits;
        const int qbi = (1 << (B - 1)) - 1;
        const uint32_t fmask = (1u << B) - 1u;
        if constexpr (OP == TileOp::Load || OP == TileOp::Import) {
            uint32_t word = 0;
            for (int s = 0; s < gr.nslot; ++s) {
                const int p = gr.p0 + s;
                if (p >= gr.pend) break;
                const int i = perm[p];
                for (int e = 0; e < 4; ++e) {
                    const int j = j0 + e;
                    int code;
                    if constexpr (OP == TileOp::Load) {
                        const float x = a.state[(tdk + i) * dv + j];
                        const float rc = a.r_in[tdk + i] * a.c_in[tdv + j];
                        float y = __builtin_rintf((x * static_cast<float>(qbi)) / rc);
                        y = fminf(fmaxf(y, -static_cast<float>(qbi)), static_cast<float>(qbi));
                        code = static_cast<int>(y);
                    } else {
                        code = a.codes_in[(tdk + i) * dv + j];
                    }
                    word |= (static_cast<uint32_t>(code) & fmask) << (8 * e + s * B);
                }
            }
            codes[d] = word;
        } else {
            const uint32_t word = codes[d];
            for (int s = 0; s < gr.nslot; ++s) {
                const int p = gr.p0 + s;
                if (p >= gr.pend) break;
                const int i = perm[p];
                for (int e = 0; e < 4; ++e) {
                    const int j = j0 + e;
                    int f = static_cast<int>((word >> (8 * e + s * B)) & fmask);
                    if (f > qbi) f -= (1 << B);
                    if constexpr (OP == TileOp::Export) {
                        a.codes_out[(tdk + i) * dv + j] = static_cast<int8_t>(f);
                    } else {
                        a.deq_out[(tdk + i) * dv + j] = (rr[p] * cc[j]) * (static_cast<float>(f) / static_cast<float>(qbi));
                    }
                }
            }
        }
    }
}

template <bool BF16, bool DIAG>
hipError_t launch_decode_128(const DecodeArgs &a, int layout, unsigned grid, hipStream_t s)
{
    switch (layout) {
    case 1: hipLaunchKernelGGL((decode_kernel<128, BF16, 1, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((decode_kernel<128, BF16, 2, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((decode_kernel<128, BF16, 3, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((decode_kernel<128, BF16, 4, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    case 5: hipLaunchKernelGGL((decode_kernel<128, BF16, 5, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((decode_kernel<128, BF16, 0, DIAG>), dim3(grid), dim3(256), 0, s, a); break;
    }
    return hipGetLastError();
}

template <bool BF16, bool DIAG>
hipError_t launch_decode_any(const DecodeArgs &a, int layout, unsigned grid, hipStream_t s)
{
    if (a.pool.dv == 128) return launch_decode_128<BF16, DIAG>(a, layout, grid, s);
    hipLaunchKernelGGL((decode_kernel<64, BF16, 0, DIAG>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const DecodeArgs &a, bool bf16, bool diag, int pool_layout, hipStream_t stream)
{
    const unsigned grid = static_cast<unsigned>(a.batch) * static_cast<unsigned>(a.pool.Hv);
    if (grid == 0) return hipSuccess;
    if (bf16) return diag ? launch_decode_any<true, true>(a, pool_layout, grid, stream)
                          : launch_decode_any<true, false>(a, pool_layout, grid, stream);
    return diag ? launch_decode_any<false, true>(a, pool_layout, grid, stream)
                : launch_decode_any<false, false>(a, pool_layout, grid, stream);
}

hipError_t launch_tile_op(const TileArgs &a, TileOp op, hipStream_t stream)
{
    const unsigned grid = static_cast<unsigned>(a.n) * static_cast<unsigned>(a.pool.Hv);
    if (grid == 0) return hipSuccess;
    switch (op) {
    case TileOp::Load: hipLaunchKernelGGL(tile_kernel<TileOp::Load>, dim3(grid), dim3(256), 0, stream, a); break;
    case TileOp::Import: hipLaunchKernelGGL(tile_kernel<TileOp::Import>, dim3(grid), dim3(256), 0, stream, a); break;
    case TileOp::Export: hipLaunchKernelGGL(tile_kernel<TileOp::Export>, dim3(grid), dim3(256), 0, stream, a); break;
    case TileOp::Dequant: hipLaunchKernelGGL(tile_kernel<TileOp::Dequant>, dim3(grid), dim3(256), 0, stream, a); break;
    }
    return hipGetLastError();
}

}  // namespace stepq
