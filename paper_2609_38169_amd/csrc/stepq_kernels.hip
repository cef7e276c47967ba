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

__device__ __forceinline__ float wave_sum(float x)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}

template <int B>
__device__ __forceinline__ void accumulate(uint32_t w, int x0, const float *s_kt, const float *s_qt,
                                           float (&acK)[4], float (&acQ)[4])
{
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float kt = s_kt[x0 + s];
        const float qt = s_qt[x0 + s];
        const uint32_t W = slot_top<B>(w, s);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float U = sbyte(W, e);
            acK[e] = fmaf(kt, U, acK[e]);
            acQ[e] = fmaf(qt, U, acQ[e]);
        }
    }
}

template <int B>
__device__ __forceinline__ uint32_t requant(uint32_t w, int x0, const float *s_al, const float *s_a,
                                            const float (&bc)[4])
{
    constexpr float qb = static_cast<float>((1 << (B - 1)) - 1);
    constexpr uint32_t fmask = (1u << B) - 1u;
    uint32_t out = 0;
#pragma unroll
    for (int s = 0; s < 8 / B; ++s) {
        const float al = s_al[x0 + s];
        const float av = s_a[x0 + s];
        const uint32_t W = slot_top<B>(w, s);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float U = sbyte(W, e);
            float y = fmaf(al, U, av * bc[e]);
            y = __builtin_rintf(y);
            y = fminf(fmaxf(y, -qb), qb);
            const uint32_t f = static_cast<uint32_t>(static_cast<int>(y)) & fmask;
            out |= f << (8 * e + s * B);
        }
    }
    return out;
}

template <int DV, bool BF16>
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a)
{
    constexpr int CG = DV / 4;              // words per row group
    constexpr int NSL = 256 / CG;           // threads sharing one column word
    constexpr int MMAX = kMaxDk * CG / 256; // words per thread when every row is 8-bit

    __shared__ float s_kt[kSlotTable], s_qt[kSlotTable], s_a[kSlotTable], s_al[kSlotTable];
    __shared__ float4 s_red[2][NSL][CG];
    __shared__ float s_b[DV];
    __shared__ float s_kap[4];

    const PoolView &P = a.pool;
    const int tid = threadIdx.x;
    const int ntiles = a.batch * P.Hv;
    const int tile = xcd_tile(blockIdx.x, ntiles);
    const int b = tile / P.Hv;
    const int h = tile - b * P.Hv;
    const int hq = h / (P.Hv / P.Hqk);
    const HeadInfo hi = P.heads[h];
    const int slot = a.slot_ids[b];
    uint8_t *rec = P.base + static_cast<uint64_t>(slot) * P.slot_bytes + hi.tile_off;
    uint32_t *codes = reinterpret_cast<uint32_t *>(rec);
    const float *rr = reinterpret_cast<const float *>(rec + hi.r_off);
    const float *cc = rr + P.dk;

    const int cg = tid % CG;
    const int slice = tid / CG;
    const int ngroups = static_cast<int>(hi.groups);

    // 1. the thread's code words (streamed: read once, written once)
    uint32_t w[MMAX];
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
        const int g = slice + NSL * m;
        w[m] = g < ngroups ? __builtin_nontemporal_load(codes + tid + 256 * m) : 0u;
    }

    // 2. per-row constants, indexed by row-table slot
    const float alpha = act_ld<BF16>(a.alpha, tile);
    const float beta = act_ld<BF16>(a.beta, tile);
    float kq = 0.f;
    if (tid < kSlotTable) {
        const int x = tid;
        int bw = 0, p = -1;
        if (x < hi.n8) {
            bw = 8;
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
            const int i = P.perm[h * P.dk + p];
            const size_t qk_off = (static_cast<size_t>(b) * P.Hqk + hq) * P.dk + i;
            const float ki = act_ld<BF16>(a.k, qk_off);
            const float qi = act_ld<BF16>(a.q, qk_off);
            const float rp = rr[p];
            const float qb = static_cast<float>((1 << (bw - 1)) - 1);
            const float fsc = 1.0f / static_cast<float>(1 << (8 - bw));
            const float rs = rp * fsc / qb;
            kt = ki * rs;
            qt = qi * rs;
            av = beta * ki * (qb / rp);
            al = alpha * fsc;
            kq = qi * ki;
        }
        s_kt[x] = kt;
        s_qt[x] = qt;
        s_a[x] = av;
        s_al[x] = al;
    }
    kq = wave_sum(kq);
    if ((tid & 63) == 0) s_kap[tid >> 6] = kq;
    __syncthreads();
    const float kappa = (s_kap[0] + s_kap[1]) + (s_kap[2] + s_kap[3]);

    // 3. S^T k and S^T q partial sums over the thread's rows, 4 columns
    float acK[4] = {0.f, 0.f, 0.f, 0.f}, acQ[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
        const int g = slice + NSL * m;
        if (g < ngroups) {
            const GroupRows gr = group_rows(hi, g);
            if (gr.bits == 8) accumulate<8>(w[m], gr.x0, s_kt, s_qt, acK, acQ);
            else if (gr.bits == 4) accumulate<4>(w[m], gr.x0, s_kt, s_qt, acK, acQ);
            else accumulate<2>(w[m], gr.x0, s_kt, s_qt, acK, acQ);
        }
    }
    s_red[0][slice][cg] = make_float4(acK[0], acK[1], acK[2], acK[3]);
    s_red[1][slice][cg] = make_float4(acQ[0], acQ[1], acQ[2], acQ[3]);
    __syncthreads();

    // 4. column reductions, residual, readout, code-space column factor
    if (tid < DV) {
        const int j = tid;
        const float *rk = reinterpret_cast<const float *>(&s_red[0][0][0]);
        const float *rq = reinterpret_cast<const float *>(&s_red[1][0][0]);
        float sk = 0.f, sq = 0.f;
#pragma unroll
        for (int s = 0; s < NSL; ++s) {
            sk += rk[s * DV + j];
            sq += rq[s * DV + j];
        }
        const float cj = cc[j];
        const float u = cj * sk;
        const float pq = cj * sq;
        const float vj = act_ld<BF16>(a.v, static_cast<size_t>(tile) * DV + j);
        const float delta = vj - alpha * u;
        a.o[static_cast<size_t>(tile) * DV + j] = alpha * pq + beta * kappa * delta;
        s_b[j] = delta / cj;
    }
    __syncthreads();

    // 5. requantize in place
    const float4 b4 = *reinterpret_cast<const float4 *>(&s_b[4 * cg]);
    const float bc[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
        const int g = slice + NSL * m;
        if (g < ngroups) {
            const GroupRows gr = group_rows(hi, g);
            uint32_t nw;
            if (gr.bits == 8) nw = requant<8>(w[m], gr.x0, s_al, s_a, bc);
            else if (gr.bits == 4) nw = requant<4>(w[m], gr.x0, s_al, s_a, bc);
            else nw = requant<2>(w[m], gr.x0, s_al, s_a, bc);
            __builtin_nontemporal_store(nw, codes + tid + 256 * m);
        }
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

}  // namespace

hipError_t launch_decode(const DecodeArgs &a, bool bf16, hipStream_t stream)
{
    const unsigned grid = static_cast<unsigned>(a.batch) * static_cast<unsigned>(a.pool.Hv);
    if (grid == 0) return hipSuccess;
    if (a.pool.dv == 128) {
        if (bf16) hipLaunchKernelGGL((decode_kernel<128, true>), dim3(grid), dim3(256), 0, stream, a);
        else hipLaunchKernelGGL((decode_kernel<128, false>), dim3(grid), dim3(256), 0, stream, a);
    } else {
        if (bf16) hipLaunchKernelGGL((decode_kernel<64, true>), dim3(grid), dim3(256), 0, stream, a);
        else hipLaunchKernelGGL((decode_kernel<64, false>), dim3(grid), dim3(256), 0, stream, a);
    }
    return hipGetLastError();
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
