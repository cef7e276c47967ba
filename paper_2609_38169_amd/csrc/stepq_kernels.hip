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
// wavefront's load covers two whole 128-byte groups.  In the compiled
// (uniform-layout) bodies the two sums over i run on the matrix cores, as
// 4x4x4 binary16 products over the 16 rows a thread holds (decode_uniform);
// the generic bodies accumulate them with v_fma_mix.  Per-column partial
// sums of the 8 threads that share a column meet in LDS; one pass over the
// words kept in registers then rewrites the codes in place.
//
// tile_kernel: pack (from fp32 states or raw codes), unpack and dequantize
// whole tiles; not on the decode path.
#include "stepq_device.h"

namespace stepq {
namespace {

// Rows of one width per word-step; codes stay in registers between passes.
// Each thread holds 16 rows (its slice's) of 4 columns; the two
// matrix-vector products run on the matrix cores as 4x4x4 blocks of 4
// threads that share their rows: A = the rows' k and q weights split into
// binary16 hi + lo parts (4 types), B = the old codes of the 4 threads'
// columns, so each thread receives the 4 weighted sums of its column.
// PIV: a padded pivot head (up to kCompactPivots FP16 pivot rows beside
// the padded uniform mix; t.hi holds its row counts and pivot offset).
template <bool BF16, bool DIAG, int M8, int M4, int M2, bool PIV = false>
__device__ __forceinline__ void decode_uniform(const DecodeArgs &a, const TileCtx &t, DecodeShared<128> &sh)
{
    constexpr int M = M8 + M4 + M2;
    static_assert(M8 + 2 * M4 + 4 * M2 == 16, "a uniform body holds 16 rows per thread");
    static_assert(M8 % 4 == 0 && M4 % 2 == 0, "row groups of 4 hold rows of one width");
    constexpr int X4 = 8 * M8, X2 = 8 * M8 + 16 * M4;    // row-table starts of the 4- and 2-bit slots
    const int tid = threadIdx.x;
    const int cg = tid & 31, slice = tid >> 5;
    const CodeWords cw(t.codes, 1024u * M);
    uint32_t w[M];
#pragma unroll
    for (int m = 0; m < M; ++m) w[m] = cw.load_m(tid, m);
    PivotRegs<128, kCompactPivots> pr;
    if constexpr (PIV) pivot_load<128, kCompactPivots>(t, slice, cg, pr);

    const RowColOps op = load_ops<BF16, DIAG, 128>(a, t.tile, t.b, t.hq, t.h, t.rr, t.cc);
    int ek, eq;
    float kappa;
    if constexpr (PIV)
        kappa = row_constants_mfma_piv<DIAG, M8, M4, M2, 128, true>(t.hi, t.alpha, t.beta, op, sh, a.pool.lv, ek, eq);
    else
        kappa = row_constants_mfma<DIAG, M8, M4, M2, 128, true>(t.beta, op, sh, a.pool.lv, ek, eq);

    uint32_t Ub[4][4][2];
    unpack_row_pairs<M8, M4, M2>(w, Ub);
    __syncthreads();    // operand table written
    matvec_partials(sh, slice, cg, Ub, ek, eq);
    if constexpr (PIV) pivot_partials_slice(t, slice, cg, pr, sh);

    column_sums<128>(a, t.tile, DIAG ? 1.0f : t.alpha, t.beta, sh, kappa, op.c, op.v);

    const float4 b4 = *reinterpret_cast<const float4 *>(&sh.bcol[4 * cg]);
    const float bc[4] = {b4.x, b4.y, b4.z, b4.w};
    if constexpr (PIV) pivot_update<128, kCompactPivots>(t, slice, cg, pr, sh, bc);
#pragma unroll
    for (int m = 0; m < M8; ++m)
        cw.store_m(tid, m, requant_word_p<8, DIAG>(Ub, m, sh.av, sh.al, slice + 8 * m, t.alpha, bc));
#pragma unroll
    for (int m = 0; m < M4; ++m)
        cw.store_m(tid, M8 + m, requant_word_p<4, DIAG>(Ub, M8 + 2 * m, sh.av, sh.al, X4 + 2 * (slice + 8 * m),
                                                        t.alpha * (1.0f / 16.0f), bc));
#pragma unroll
    for (int m = 0; m < M2; ++m)
        cw.store_m(tid, M8 + M4 + m,
                   requant_word_p<2, DIAG>(Ub, M8 + 2 * M4 + 4 * m, sh.av, sh.al, X2 + 4 * (slice + 8 * m),
                                           t.alpha * (1.0f / 64.0f), bc));
}

// Any row-width mix and d_v: the class of each word-step is looked up at run
// time and the words are unpacked again for the second pass.  MMAX word-steps
// (row groups / NSL) and PMAX pivot rows per head at most.
template <bool BF16, bool DIAG, int DV, int MMAX, int PMAX>
__device__ __forceinline__ void decode_generic(const DecodeArgs &a, const TileCtx &t, DecodeShared<DV> &sh)
{
    constexpr int CG = DV / 4;
    constexpr int NSL = 256 / CG;
    const int tid = threadIdx.x;
    const int cg = tid % CG, slice = tid / CG;
    const int ngroups = static_cast<int>(t.hi.groups);
    // words of groups past the head's last lie in the zeroed tail of the
    // codes region or past it (read as 0): one uniform check per word-step
    const CodeWords cw(t.codes, t.hi.piv_off);
    uint32_t w[MMAX];
#pragma unroll
    for (int m = 0; m < MMAX; ++m) w[m] = NSL * m < ngroups ? cw.load(tid + 256 * m) : 0u;
    PivotRegs<DV, PMAX> pr;
    pivot_load(t, slice, cg, pr);
    const RowColOps op = load_ops<BF16, DIAG, DV>(a, t.tile, t.b, t.hq, t.h, t.rr, t.cc);
    const float kappa = row_constants<DIAG, DV, true>(t.hi, a.pool.dk, t.alpha, t.beta, op, sh, a.pool.lv);

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
    pivot_acc(t, slice, cg, pr, sh, acK, acQ);
    column_phase<DV>(a, t.tile, DIAG ? 1.0f : t.alpha, t.beta, sh, kappa, acK, acQ, op.c, op.v);

    const float4 b4 = *reinterpret_cast<const float4 *>(&sh.bcol[4 * cg]);
    const float bc[4] = {b4.x, b4.y, b4.z, b4.w};
    pivot_update(t, slice, cg, pr, sh, bc);
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
            cw.store(tid + 256 * m, nw);
        }
    }
}

// A head at d = 128 whose integer rows are 8- and 4-bit in any split, in the
// compact layout, with up to kCompactPivots FP16 pivot rows (the per-row
// maps of a row-unit calibration).  Groups below hi.g8 are 8-bit, the rest
// up to hi.groups 4-bit, so a word-step's width changes between slices at
// most once.  Both sums over rows run on the matrix cores: per word group
// of 4 word-steps, a 4x4x4 block per column for the words' slot-0 view and,
// where the group holds 4-bit words, one for their slot-1 view.  The
// requantization reads the fields again from the words kept in registers.
template <bool BF16, bool DIAG>
__device__ __forceinline__ void decode_rowmix(const DecodeArgs &a, const TileCtx &t, DecodeShared<128> &sh)
{
    const int tid = threadIdx.x;
    const int cg = tid & 31, slice = tid >> 5;
    const int g8 = __builtin_amdgcn_readfirstlane(static_cast<int>(t.hi.g8));
    const int ng = __builtin_amdgcn_readfirstlane(static_cast<int>(t.hi.groups));
    // the buffer covers the codes region only (piv_off = 128 ng): the words
    // of groups past the head's last read 0 and their stores are dropped, so
    // each word-step needs one uniform check and no per-lane one
    const CodeWords cw(t.codes, t.hi.piv_off);
    uint32_t w[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) w[m] = 8 * m < ng ? cw.load(tid + 256 * m) : 0u;
    PivotRegs<128, kCompactPivots> pr;
    pivot_load<128, kCompactPivots>(t, slice, cg, pr);
    const RowColOps op = load_ops<BF16, DIAG, 128>(a, t.tile, t.b, t.hq, t.h, t.rr, t.cc);
    rowmix_sums<DIAG, true, true>(a, t, sh, w, pr, op, g8, ng);

    const float4 b4 = *reinterpret_cast<const float4 *>(&sh.bcol[4 * cg]);
    const float bc[4] = {b4.x, b4.y, b4.z, b4.w};
    pivot_update<128, kCompactPivots>(t, slice, cg, pr, sh, bc);
    // row-table slot of group g: g when 8-bit, c4 + 2 g (= g8 + 2 (g - g8))
    // when 4-bit; word-steps wholly of one width take a uniform path, the one
    // straddling the width boundary a per-lane one
    const int c4 = -g8;
    const float al4 = t.alpha * (1.0f / 16.0f);
    float U[8];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
        const int g = slice + 8 * m;
        if (8 * m >= ng) break;
        if (8 * m + 8 <= g8) {
            unpack_word<8>(w[m], U);
            cw.store(tid + 256 * m, requant_word<8, DIAG>(U, sh.av, sh.al, g, t.alpha, bc));
        } else if (8 * m >= g8) {
            // lanes past the head's last group read table entries of other
            // rows, and their stores are dropped
            unpack_word<4>(w[m], U);
            cw.store(tid + 256 * m, requant_word<4, DIAG>(U, sh.av, sh.al, c4 + 2 * g, al4, bc));
        } else if (g < g8) {
            unpack_word<8>(w[m], U);
            cw.store(tid + 256 * m, requant_word<8, DIAG>(U, sh.av, sh.al, g, t.alpha, bc));
        } else {
            unpack_word<4>(w[m], U);
            cw.store(tid + 256 * m, requant_word<4, DIAG>(U, sh.av, sh.al, c4 + 2 * g, al4, bc));
        }
    }
}

template <bool BF16, bool DIAG, int L>
__device__ __forceinline__ void run_uniform(const DecodeArgs &a, TileCtx &t, int slot, DecodeShared<128> &sh)
{
    // every tile record of layout L is (codes: 1024 bytes per word-step) + r + c
    constexpr UniformLayout u = kUniformLayouts[L - 1];
    constexpr uint32_t r_off = 1024u * (u.m8 + u.m4 + u.m2);
    uint8_t *rec = a.pool.base + static_cast<uint64_t>(slot) * a.pool.slot_bytes + t.off;
    t.codes = reinterpret_cast<uint32_t *>(rec);
    t.rr = reinterpret_cast<const float *>(rec + r_off);
    t.cc = t.rr + 128;
    decode_uniform<BF16, DIAG, u.m8, u.m4, u.m2>(a, t, sh);
}

// A padded pivot head of uniform layout L: codes (1024 bytes per
// word-step), the n16 pivot rows (256 bytes each), r, c; its row counts
// come from the head list.
template <bool BF16, bool DIAG, int L>
__device__ __forceinline__ void run_uniform_piv(const DecodeArgs &a, TileCtx &t, int slot, DecodeShared<128> &sh)
{
    constexpr UniformLayout u = kUniformLayouts[L - 1];
    padded_pivot_tile<L>(a, t, slot);
    decode_uniform<BF16, DIAG, u.m8, u.m4, u.m2, true>(a, t, sh);
}

template <bool BF16, bool DIAG>
__device__ __forceinline__ void run_rowmix(const DecodeArgs &a, TileCtx &t, int slot, DecodeShared<128> &sh)
{
    const PoolView &P = a.pool;
    t.hi = P.heads[t.h];
    uint8_t *rec = P.base + static_cast<uint64_t>(slot) * P.slot_bytes + t.hi.tile_off;
    t.codes = reinterpret_cast<uint32_t *>(rec);
    t.rr = reinterpret_cast<const float *>(rec + t.hi.r_off);
    t.cc = t.rr + 128;
    decode_rowmix<BF16, DIAG>(a, t, sh);
}

template <bool BF16, bool DIAG, int DV, bool COMPACT>
__device__ __forceinline__ void run_generic(const DecodeArgs &a, TileCtx &t, int slot, DecodeShared<DV> &sh)
{
    const PoolView &P = a.pool;
    t.hi = P.heads[t.h];
    uint8_t *rec = P.base + static_cast<uint64_t>(slot) * P.slot_bytes + t.hi.tile_off;
    t.codes = reinterpret_cast<uint32_t *>(rec);
    t.rr = reinterpret_cast<const float *>(rec + t.hi.r_off);
    t.cc = t.rr + P.dk;
    constexpr int full_m = kMaxDk * (DV / 4) / 256;
    decode_generic<BF16, DIAG, DV, COMPACT ? kCompactGroups / 8 : full_m, COMPACT ? kCompactPivots : kMaxPivots>(
        a, t, sh);
}

// LAYOUT in 1 .. kNumUniformLayouts: every head of the launch has that
// uniform layout (the host launches each layout class of a pool
// separately), so the kernel holds only that body and its register budget.
// LAYOUT == 0: the generic body (irregular row-width mixes, FP16 pivot
// rows, d_v = 64).  LAYOUT == kCompactGeneric: the generic body for heads of
// at most kCompactGroups row groups and kCompactPivots pivot rows (d_v =
// 128), in fewer registers.  LAYOUT == kMixedBase + L: heads of uniform
// layout L and compact generic heads in one launch, told apart by the head
// list (both bodies fit the same register budget), together with layout-L
// padded pivot heads; kMixedF16Base + L: the same with whole FP16 heads too.
// LAYOUT == kMultiUniform: heads of several compiled layouts (uniform,
// whole FP16), each tile dispatched to its own body; kMultiPivot: with
// padded pivot heads too.
// LAYOUT == kRowMix: compact heads of 8- and 4-bit rows in any split with at
// most kCompactPivots pivot rows (decode_rowmix), launched as a class of its
// own (in the combined launches it would raise their register count).
// LAYOUT == kMixedPivotBase + L: uniform layout-L heads and layout-L padded
// pivot heads only.  LAYOUT == kPivotUniformBase + L: padded pivot heads of
// uniform layout L only.  LAYOUT == kF16HeadLayout: heads held entirely in FP16 (every mode;
// the host sets a.f16_c_one for the row-absmax step).
template <int DV, bool BF16, int LAYOUT, bool DIAG>
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a)
{
    __shared__ DecodeShared<DV> sh;
    TileCtx t;
    uint32_t tile_bytes = 0;
    if constexpr (DV == 128 && LAYOUT > 0 && LAYOUT <= kNumUniformLayouts) {
        constexpr UniformLayout u = kUniformLayouts[LAYOUT - 1];
        tile_bytes = 1024u * (u.m8 + u.m4 + u.m2 + 1);
    } else if constexpr (DV == 128 && LAYOUT == kF16HeadLayout) {
        tile_bytes = 128u * 256u + 1024u;
    }
    tile_of(a, tile_bytes, t);
    const int slot = a.slot_ids[t.b];
    t.alpha = DIAG ? 1.0f : act_ld<BF16>(a.alpha, t.tile);
    t.beta = act_ld<BF16>(a.beta, t.tile);
    if constexpr (DV == 128 && (LAYOUT == kMultiUniform || LAYOUT == kMultiPivot)) {
        switch (t.layout) {
        case 1: run_uniform<BF16, DIAG, 1>(a, t, slot, sh); break;
        case 2: run_uniform<BF16, DIAG, 2>(a, t, slot, sh); break;
        case 3: run_uniform<BF16, DIAG, 3>(a, t, slot, sh); break;
        case 4: run_uniform<BF16, DIAG, 4>(a, t, slot, sh); break;
        case 5: run_uniform<BF16, DIAG, 5>(a, t, slot, sh); break;
        case kF16HeadLayout: run_f16head<BF16, DIAG>(a, t, slot, sh); break;
        default:
            if constexpr (LAYOUT == kMultiPivot) {
                switch (t.layout - kPivotUniformBase) {
                case 1: run_uniform_piv<BF16, DIAG, 1>(a, t, slot, sh); break;
                case 2: run_uniform_piv<BF16, DIAG, 2>(a, t, slot, sh); break;
                case 3: run_uniform_piv<BF16, DIAG, 3>(a, t, slot, sh); break;
                case 4: run_uniform_piv<BF16, DIAG, 4>(a, t, slot, sh); break;
                default: run_uniform_piv<BF16, DIAG, 5>(a, t, slot, sh); break;
                }
            }
            break;
        }
    } else if constexpr (DV == 128 && LAYOUT == kRowMix) {
        run_rowmix<BF16, DIAG>(a, t, slot, sh);
    } else if constexpr (DV == 128 && LAYOUT > 0 && LAYOUT <= kNumUniformLayouts) {
        run_uniform<BF16, DIAG, LAYOUT>(a, t, slot, sh);
    } else if constexpr (DV == 128 && LAYOUT == kF16HeadLayout) {
        run_f16head<BF16, DIAG>(a, t, slot, sh);
    } else if constexpr (DV == 128 && LAYOUT > kPivotUniformBase) {
        run_uniform_piv<BF16, DIAG, LAYOUT - kPivotUniformBase>(a, t, slot, sh);
    } else if constexpr (DV == 128 && LAYOUT > kMixedPivotBase) {
        // one body for both: a layout-L head is a padded pivot head with no pivot rows
        run_uniform_piv<BF16, DIAG, LAYOUT - kMixedPivotBase>(a, t, slot, sh);
    } else if constexpr (DV == 128 && LAYOUT > kMixedF16Base) {
        constexpr int L = LAYOUT - kMixedF16Base;
        if (t.layout == L) {
            run_uniform<BF16, DIAG, L>(a, t, slot, sh);
        } else if (t.layout == kPivotUniformBase + L) {
            run_uniform_piv<BF16, DIAG, L>(a, t, slot, sh);
        } else if (t.layout == kF16HeadLayout) {
            run_f16head<BF16, DIAG>(a, t, slot, sh);
        } else {
            run_generic<BF16, DIAG, 128, true>(a, t, slot, sh);
        }
    } else if constexpr (DV == 128 && LAYOUT > kMixedBase) {
        constexpr int L = LAYOUT - kMixedBase;
        if (t.layout == L) run_uniform<BF16, DIAG, L>(a, t, slot, sh);
        else if (t.layout == kPivotUniformBase + L) run_uniform_piv<BF16, DIAG, L>(a, t, slot, sh);
        else run_generic<BF16, DIAG, 128, true>(a, t, slot, sh);
    } else {
        run_generic<BF16, DIAG, DV, DV == 128 && LAYOUT == kCompactGeneric>(a, t, slot, sh);
    }
}

// ---------------------------------------------------------------------------
// Memory-only reference of the decode step (a measurement aid, not part of
// the method): the same tiles in the same workgroup order (tile_of), each
// thread reading the same code words with the same policy (non-temporal
// loads, all issued before any store) and writing them back unchanged
// (sc1 nt stores), the scales read once, the activations read and o
// written; no arithmetic.  `zero` is 0 at run time: the XOR keeps the
// compiler from dropping a store of a value just loaded from the same
// address, and o receives zeros.
template <bool BF16>
__global__ __launch_bounds__(256) void stream_ref_kernel(DecodeArgs a, uint32_t zero)
{
    const PoolView &P = a.pool;
    TileCtx t;
    tile_of(a, 0u, t);
    const HeadInfo hi = P.heads[t.h];
    const int slot = a.slot_ids[t.b];
    uint8_t *rec = P.base + static_cast<uint64_t>(slot) * P.slot_bytes + hi.tile_off;
    const int tid = threadIdx.x;
    // codes and pivot rows: everything before r
    const CodeWords cw(rec, hi.r_off);
    const int nw = static_cast<int>(hi.r_off / 4);
    constexpr int kMaxWords = 32;          // a whole FP16 head: 32 KiB = 32 words per thread
    uint32_t w[kMaxWords];
#pragma unroll
    for (int m = 0; m < kMaxWords; ++m) w[m] = 256 * m < nw ? cw.load(tid + 256 * m) : 0u;
    const float *rr = reinterpret_cast<const float *>(rec + hi.r_off);
    float acc = 0.f;
    if (tid < P.dk) {
        acc += rr[tid];
        const size_t off = (static_cast<size_t>(t.b) * P.Hqk + t.hq) * P.dk + tid;
        acc += act_ld<BF16>(a.k, off) + act_ld<BF16>(a.q, off);
    }
    if (tid < P.dv) acc += rr[P.dk + tid] + act_ld<BF16>(a.v, static_cast<size_t>(t.tile) * P.dv + tid);
    acc += act_ld<BF16>(a.alpha, t.tile) + act_ld<BF16>(a.beta, t.tile);
#pragma unroll
    for (int m = 0; m < kMaxWords; ++m)
        if (256 * m < nw) cw.store(tid + 256 * m, w[m] ^ zero);
    if (tid < P.dv) a.o[static_cast<size_t>(t.tile) * P.dv + tid] = acc * __uint_as_float(zero);
}

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
        for (uint32_t d = hi.groups * CG + tid; d < hi.piv_off / 4; d += 256) rec32[d] = 0u;
        for (uint32_t d = (hi.r_off + 4u * (dk + dv)) / 4 + tid; d < hi.tile_bytes / 4; d += 256) rec32[d] = 0u;
    }
    if constexpr (OP == TileOp::Export) {
        for (int p = tid; p < dk; p += 256) a.r_out[tdk + perm[p]] = rr[p];
        for (int j = tid; j < dv; j += 256) a.c_out[tdv + j] = cc[j];
    }

    // FP16 pivot rows: physical rows 0 .. n16-1, d_v binary16 values each
    uint16_t *piv = reinterpret_cast<uint16_t *>(rec + hi.piv_off);
    const int npv = static_cast<int>(hi.n16) * dv;
    if constexpr (OP == TileOp::ExportPivots || OP == TileOp::ImportPivots) {
        for (int e = tid; e < dk * dv; e += 256) {
            const int p = e / dv, j = e - p * dv;
            const size_t o = (tdk + perm[p]) * dv + j;
            if constexpr (OP == TileOp::ExportPivots) a.piv_out[o] = p < hi.n16 ? piv[e] : static_cast<uint16_t>(0);
            else if (p < hi.n16) piv[e] = a.piv_in[o];
        }
        return;
    } else {
        for (int e = tid; e < npv; e += 256) {
            const int p = e / dv, j = e - p * dv;
            const size_t o = (tdk + perm[p]) * dv + j;
            if constexpr (OP == TileOp::Load)
                piv[e] = __builtin_bit_cast(uint16_t, static_cast<_Float16>(a.state[o]));    // nearest even
            else if constexpr (OP == TileOp::Export)
                a.codes_out[o] = 0;
            else if constexpr (OP == TileOp::Dequant)
                a.deq_out[o] = static_cast<float>(__builtin_bit_cast(_Float16, piv[e]));
        }
    }

    const int nw = static_cast<int>(hi.groups) * CG;
    for (int d = tid; d < nw; d += 256) {
        const int g = d / CG;
        const int j0 = 4 * (d - g * CG);
        const GroupRows gr = group_rows(hi, g);
        const int B = gr.bits;
        const int qbi = (1 << (B - 1)) - 1;
        const float iq = P.lv.iq[B == 8 ? 0 : (B == 4 ? 1 : 2)];     // q = level * iq
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
                        float y = __builtin_rintf((x * iq) / rc);
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
                        a.deq_out[(tdk + i) * dv + j] = (rr[p] * cc[j]) * (static_cast<float>(f) / iq);
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
    case kCompactGeneric:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kCompactGeneric, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kF16HeadLayout:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kF16HeadLayout, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kPivotUniformBase + 1:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kPivotUniformBase + 1, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kPivotUniformBase + 2:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kPivotUniformBase + 2, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kPivotUniformBase + 3:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kPivotUniformBase + 3, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kPivotUniformBase + 4:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kPivotUniformBase + 4, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kPivotUniformBase + 5:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kPivotUniformBase + 5, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kMultiUniform:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kMultiUniform, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kMultiPivot:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kMultiPivot, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kRowMix:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kRowMix, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kMixedPivotBase + 1:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kMixedPivotBase + 1, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kMixedPivotBase + 2:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kMixedPivotBase + 2, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kMixedBase + 1:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kMixedBase + 1, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kMixedBase + 2:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kMixedBase + 2, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kMixedF16Base + 1:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kMixedF16Base + 1, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
    case kMixedF16Base + 2:
        hipLaunchKernelGGL((decode_kernel<128, BF16, kMixedF16Base + 2, DIAG>), dim3(grid), dim3(256), 0, s, a);
        break;
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
    const unsigned grid = static_cast<unsigned>(a.batch) * static_cast<unsigned>(a.n_heads);
    if (grid == 0) return hipSuccess;
    if (bf16) return diag ? launch_decode_any<true, true>(a, pool_layout, grid, stream)
                          : launch_decode_any<true, false>(a, pool_layout, grid, stream);
    return diag ? launch_decode_any<false, true>(a, pool_layout, grid, stream)
                : launch_decode_any<false, false>(a, pool_layout, grid, stream);
}

hipError_t launch_stream_ref(const DecodeArgs &a, bool bf16, hipStream_t stream)
{
    const unsigned grid = static_cast<unsigned>(a.batch) * static_cast<unsigned>(a.n_heads);
    if (grid == 0) return hipSuccess;
    if (bf16) hipLaunchKernelGGL(stream_ref_kernel<true>, dim3(grid), dim3(256), 0, stream, a, 0u);
    else hipLaunchKernelGGL(stream_ref_kernel<false>, dim3(grid), dim3(256), 0, stream, a, 0u);
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
    case TileOp::ExportPivots:
        hipLaunchKernelGGL(tile_kernel<TileOp::ExportPivots>, dim3(grid), dim3(256), 0, stream, a);
        break;
    case TileOp::ImportPivots:
        hipLaunchKernelGGL(tile_kernel<TileOp::ImportPivots>, dim3(grid), dim3(256), 0, stream, a);
        break;
    }
    return hipGetLastError();
}

}  // namespace stepq
