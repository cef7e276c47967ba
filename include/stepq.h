/*
 * stepq.h -- C ABI of the MI355X (gfx950) quantized gated-Delta decode step.
 *
 * The library keeps a pool of recurrent states S in R^{d_k x d_v}, one per
 * (request slot, value head), stored as mixed-precision integer codes with
 * per-tile key-row and value-column scales, and advances the active ones by
 * one decode step in a single fused kernel launch.
 *
 * What one decode step computes (paper: Eq. 1 with the GDN gate D = alpha I,
 * Eq. 3, Eq. 4, Section 4.3 and Appendix C, Table C2, with frozen scales):
 *   S^_ij = r_i c_j q_ij / q_{b_i}                 reconstruction, q_b = 2^(b-1)-1
 *   X     = alpha S^ + beta k (v - alpha S^T k)^T   gated Delta update
 *   o     = X^T q                                  readout, taken before requantization
 *   q'_ij = clip(round(X_ij q_{b_i} / (r_i c_j)), -q_{b_i}, q_{b_i})   round = ties-to-even
 * and q' replaces q in place; r and c are left unchanged.  These are the
 * formulas of the default level normalisation N1 (stepq_levels below); under
 * N2 every q / q_b becomes 2^(8-b) q and every X q_b / (...) becomes
 * X 2^(b-8) / (...).
 *
 * Conventions for every call:
 *  - Pointers named *_dev, and every array argument of the device calls, are
 *    device memory of the current HIP device; the descriptor's tables and the
 *    setup calls' arrays are host memory.  The caller owns all of it.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Device calls only
 *    enqueue work on it and return; inputs must stay alive, and outputs must
 *    not be read, until the stream has reached the work.
 *  - A pool must not be used from two streams at once.  In one decode step
 *    the slot ids must be distinct and in [0, n_slots): each (slot, head)
 *    tile is rewritten in place by exactly one workgroup.  With the
 *    environment variable STEPQ_DEBUG=1 this is checked on the host (a
 *    synchronising copy of the ids) and violations return STEPQ_E_INVALID.
 *  - One call handles at most 2^24 (slot, head) tiles (n x n_v_heads); larger
 *    calls return STEPQ_E_UNSUPPORTED and are split by the caller.
 *  - Nothing is thrown across the ABI.  Invalid arguments return
 *    STEPQ_E_INVALID before anything is enqueued; a failing HIP call returns
 *    STEPQ_E_HIP.  stepq_last_error() describes the last failure of the
 *    calling thread.
 *
 * ---------------------------------------------------------------------------
 * Pool layout (what stepq_pool_device_ptr() points at)
 *
 * The pool is n_slots slot records of slot_bytes each, back to back.  A slot
 * record is the tile records of value heads 0 .. n_v_heads-1 in order.  The
 * tile record of head h, whose key rows have widths row_bits[h][0 .. d_k-1]
 * (each 8, 4 or 2, or 16 for an FP16 pivot row; the same for every slot, the
 * paper's fixed precision map and pivot set, Section 3.2):
 *
 *  - Physical row order: the pivot rows in increasing logical row index, then
 *    the 8-bit rows, the 4-bit rows and the 2-bit rows, each the same way.
 *    n16, n8, n4, n2 = row counts; n16 <= 32, or n16 = d_k = d_v = 128: a
 *    head held entirely in FP16 (Table C1 keeps whole heads of the GDN model
 *    as pivots).  Such a tile is its 32 KiB pivot region plus the r and c
 *    slots, which stay unused (the paper's serving layout omits them).
 *  - Row groups: each group holds 8/b physical integer rows of one width b --
 *    one 8-bit row, two 4-bit rows or four 2-bit rows -- filled in physical
 *    order.  Groups are ordered 8-bit, 4-bit, 2-bit, with G8, G4, G2 groups
 *    of each width, G = G8 + G4 + G2.  Normally G8 = n8, G4 = ceil(n4/2),
 *    G2 = ceil(n2/4), and a width's last group may have empty slots.  At
 *    d_k = d_v = 128 (whole-FP16 heads aside) the integer rows may fit one
 *    of the uniform mixes, in units of 8 groups {8-bit, 4-bit, 2-bit}:
 *    {8,4,0}, {4,2,2}, {16,0,0}, {0,8,0}, {0,0,4}.  The first mix in this
 *    order with 8 m8 >= n8, 16 m4 >= n4 and 32 m2 >= n2 then sets
 *    G8 = 8 m8, G4 = 8 m4, G2 = 8 m2: each width's rows fill its groups from
 *    the first, and the groups after them stay empty.  Without pivot rows
 *    this is exactly the tight layout; a head with pivot rows is padded to
 *    the mix, so that the compiled decode body for that mix can run it.
 *  - Codes region: G groups of d_v bytes each.  Byte j of a group holds
 *    column j of all its rows: the row in slot s (0-based, in physical
 *    order) occupies bits [s*b, s*b + b) as a b-bit two's-complement integer
 *    in [-q_b, q_b]; empty slots are 0.  The region is zero-padded to a
 *    multiple of 128 bytes.
 *  - Pivot region: the n16 pivot rows in physical order, d_v IEEE binary16
 *    values each (little-endian): 2 d_v bytes per row.
 *  - Then r: d_k fp32 row scales in physical row order (a pivot row's entry
 *    is carried but unused); then c: d_v fp32 column scales.  The record is
 *    zero-padded to a multiple of 128 bytes.
 *
 * Pivot rows hold their values directly: every step updates them like any
 * other row and stores X rounded to binary16 (nearest, ties to even); they
 * take no part in the scale fits.
 *
 * So a 6-bit tile (64 rows @8 + 64 rows @4, d = 128) is 12,288 code bytes +
 * 1,024 scale bytes = 13,312 bytes, read once and its codes written once per
 * decode step.  The code-carrying part of every group is one 128-byte line at
 * d_v = 128, so a wavefront's dword load covers two whole lines.
 */
#ifndef STEPQ_H
#define STEPQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    STEPQ_OK = 0,
    STEPQ_E_INVALID = 1,      /* bad argument; nothing was enqueued */
    STEPQ_E_UNSUPPORTED = 2,  /* well-formed but outside what the library implements */
    STEPQ_E_NOMEM = 3,        /* device allocation failed */
    STEPQ_E_HIP = 4           /* a HIP runtime call failed */
} stepq_status;

typedef enum {
    STEPQ_F32 = 0,            /* activations as float */
    STEPQ_BF16 = 1            /* activations as bfloat16 (upper half of a float) */
} stepq_dtype;

/* Level normalisation of the stored integers (Section 4.3, Appendix C.1): a
 * b-bit code q (|q| <= q_b = 2^(b-1) - 1) stands for the level z, and
 * S^_ij = r_i c_j z_ij.  Every scale fit, quantization and reconstruction of
 * a pool uses its normalisation. */
typedef enum {
    STEPQ_LEVELS_ABSMAX = 0,  /* N1: z = q / q_b, so |S^_ij| <= r_i c_j at every width (default) */
    STEPQ_LEVELS_POW2 = 1     /* N2: z = 2^(8-b) q, the paper's KDA codebook; top level 2^(8-b) q_b */
} stepq_levels;

typedef struct stepq_pool stepq_pool;   /* opaque */

typedef struct {
    int32_t n_slots;          /* >= 1 */
    int32_t n_v_heads;        /* Hv >= 1 */
    int32_t n_qk_heads;       /* Hqk >= 1, Hv % Hqk == 0; value head h reads q/k head h / (Hv/Hqk) */
    int32_t d_k;              /* key rows per tile, 1 .. 128 */
    int32_t d_v;              /* value columns per tile, 64 or 128 */
    const uint8_t *row_bits;  /* host [Hv][d_k], each 2, 4, 8 or 16 (pivot); copied by stepq_pool_create */
    int32_t levels;           /* stepq_levels; 0 (a zero-initialised descriptor) is N1 */
} stepq_pool_desc;

/* Size of the pool described by desc (layout above).  Either output may be
 * NULL.  Host only, no device work.  STEPQ_E_UNSUPPORTED when one slot
 * record would exceed 4 GiB (tile offsets inside a record are 32-bit). */
stepq_status stepq_pool_bytes(const stepq_pool_desc *desc, size_t *pool_bytes, size_t *slot_bytes);

/* One launch of a decode step (stepq_pool_plan). */
typedef struct {
    int32_t body;             /* the kernel body it runs (library-internal launch code) */
    int32_t first;            /* first position of head_order the launch covers */
    int32_t n_heads;          /* value heads it covers: its grid is batch x n_heads workgroups */
} stepq_launch_desc;

/* The kernel launches of one decode step of a pool with this descriptor and
 * these stepq_decode_step_ex flags, in launch order.  Host only, no device
 * work.  Heads of one layout class share a launch (a frozen step of a pool
 * whose classes all have a combined body is one launch); each launch covers
 * positions [first, first + n_heads) of head_order [n_v_heads] (NULL: not
 * written), which receives the value head at each position.  At most
 * max_launches entries are written to launches; *n_launches receives the
 * full count.  The plan is checked exactly as stepq_pool_create checks it:
 * each tile's records lie inside the slot record, every head is listed once
 * with its own tile offset, and each launch's body runs every head it gets.
 * Errors as stepq_pool_create (a failed plan check is STEPQ_E_INVALID). */
stepq_status stepq_pool_plan(const stepq_pool_desc *desc, uint32_t flags, stepq_launch_desc *launches,
                             int32_t max_launches, int32_t *n_launches, int32_t *head_order);

/* Create a pool.  device_mem: caller-owned device memory of at least
 * stepq_pool_bytes() bytes, 256-byte aligned, whose contents become the
 * pool; or NULL, in which case the library allocates (and later frees) it.
 * The pool contents are undefined until written by stepq_pool_load or
 * stepq_pool_import.  Allocates the small per-head layout tables on the
 * current device.  Blocks until they are copied.  The decode launches are
 * planned and checked on the host first (stepq_pool_plan); a plan that
 * fails its check returns STEPQ_E_INVALID before any allocation.
 * STEPQ_E_NOMEM when an allocation fails, STEPQ_E_HIP when a copy does. */
stepq_status stepq_pool_create(const stepq_pool_desc *desc, void *device_mem, size_t device_mem_bytes,
                               stepq_pool **out);

/* Release the pool object, its layout tables and (only if the library
 * allocated it) the pool memory.  Synchronises the device first.  NULL ok. */
void stepq_pool_destroy(stepq_pool *pool);

/* Raw pool memory (layout above), for saving, restoring or inspecting it. */
void *stepq_pool_device_ptr(const stepq_pool *pool);

/* Quantize and pack full-precision states into slots: the pack of the
 * boundary states after prefill, which hands a request's state to the
 * decode pool (Appendix F.1, the packed-state integration: prefill runs on
 * full-precision states and packs the states at its boundary).  For i < n:
 * slot slot_ids[i] receives
 *   q_hj = clip(round(state[i][h][j][:] / (r c nu)), -q_b, q_b)
 * with scales r (logical row order) and c stored alongside, nu the level
 * step of the row's width (1/q_b under N1, 2^(8-b) under N2).
 *   slot_ids [n] int32, state [n][Hv][d_k][d_v] fp32 (logical row order),
 *   r [n][Hv][d_k] fp32 > 0, c [n][Hv][d_v] fp32 > 0.
 * The rounding is taken in fp32. */
stepq_status stepq_pool_load(stepq_pool *pool, const int32_t *slot_ids, int32_t n, const float *state,
                             const float *r, const float *c, void *stream);

/* One fused decode step for `batch` active requests (the update written out
 * at the top of this header).  For b < batch, tile (slot_ids[b], h) reads
 *   q[b][h/(Hv/Hqk)][:], k[b][h/(Hv/Hqk)][:]  (d_k each),  v[b][h][:] (d_v),
 *   alpha[b][h], beta[b][h]
 * in act_dtype (arrays [batch][Hqk][d_k], [batch][Hv][d_v], [batch][Hv]),
 * writes o[b][h][:] (fp32, [batch][Hv][d_v]) and rewrites its codes in
 * place.  The arithmetic is fp32, except that in the compiled bodies of the
 * uniform row-width mixes, and of heads at d_k = d_v = 128 whose integer
 * rows are 8- and 4-bit in any split with at most 8 FP16 pivot rows (the
 * per-row maps of a row-unit calibration), S^T k and S^T q run on the
 * matrix cores: each row weight (k_i r_i / q_b, q_i r_i / q_b, scaled by a
 * power of two per tile) is split into binary16 hi + lo parts (22
 * significant bits), the codes are exact in binary16, and the products
 * accumulate in fp32.  The
 * new code's field value y = code + 2^(b-1) is formed as (y - 1) / S,
 * clamped to [0, 1] and scaled back (S = 256, 14 or 2 for 8-, 4- and 2-bit
 * fields; exact scalings except for 4-bit fields, a few ulp of values at
 * most 15), then rounded to nearest even.  With STEPQ_STEP_REFIT the gate
 * term of the unrounded code may run on a matrix-core block, within one
 * ulp of the fp32 FMA.
 * batch == 0 is a no-op. */
stepq_status stepq_decode_step(stepq_pool *pool, const int32_t *slot_ids, int32_t batch, const void *q,
                               const void *k, const void *v, const void *alpha, const void *beta,
                               stepq_dtype act_dtype, float *o, void *stream);

/* The same decode step with the channel-wise retention gate of KDA,
 * D = diag(d) instead of alpha I (paper, Section 2.1 and Eq. 1):
 *   X = D S^ + beta k (v - S^T D k)^T,   o = X^T q,
 * requantized as above.  gate: [batch][Hv][d_k] in act_dtype, one retention
 * factor per key row (logical order) of each (request, value head); the
 * other arguments are those of stepq_decode_step.  With every d_i equal to
 * alpha the two calls compute the same update. */
stepq_status stepq_decode_step_kda(stepq_pool *pool, const int32_t *slot_ids, int32_t batch, const void *q,
                                   const void *k, const void *v, const void *gate, const void *beta,
                                   stepq_dtype act_dtype, float *o, void *stream);

/* Flags of stepq_decode_step_ex. */
enum {
    STEPQ_STEP_KDA_GATE = 1u,  /* gate is the channel-wise d [batch][Hv][d_k] (KDA), else alpha [batch][Hv] */
    STEPQ_STEP_REFIT = 2u,     /* refit both scale vectors to the updated state before requantizing */
    STEPQ_STEP_ROW_ABSMAX = 4u, /* single-axis baseline: r'_i = max_j |X_ij|, c' = 1 (excludes REFIT) */
    STEPQ_STEP_ADJACENT_SLOTS = 8u /* hint: slot_ids[b] = slot_ids[0] + b (see below) */
};

/* The decode step with optional channel-wise gate and online scale refit.
 * Without STEPQ_STEP_REFIT it is stepq_decode_step (or _kda with
 * STEPQ_STEP_KDA_GATE).  With STEPQ_STEP_REFIT the stored scales of every
 * updated tile are replaced by the Key-Row-Aware Dual-Axis fit of X (paper,
 * Section 4.3, Appendix C.1 and Table C2 steps 4-6), w being the pool's
 * row-impact factors (stepq_pool_set_row_weight, default 1), as the
 * fixed-code column update of Appendix C.1 prescribes:
 *   r'_i = (m_i / w_i)^{1/2},  m_i = (1/d_v) sum_j |X_ij|
 *   c0_j = max_i |X_ij| / r'_i                     (start of the column fit)
 *   z_ij = clip(round(X_ij q_b / (r'_i c0_j)), -q_b, q_b) / q_b   (fixed codes)
 *   c'_j = c_j sum_i W_i z_ij y_ij / sum_i W_i z_ij^2,  W_i = (w_i r'_i / q_b)^2,
 *          y_ij = X_ij q_b / (r'_i c_j)
 *        = the minimiser over c of sum_i w_i^2 (X_ij - r'_i c z_ij)^2;
 *          a zero denominator keeps c_j
 *   q'_ij = clip(round(X_ij q_b / (r'_i c'_j)), -q_b, q_b)
 * r', c0 and c' are floored at 2^-60; r' and c' are written as the new fp32
 * scales.  The readout o is X^T q as without the flag.
 * With STEPQ_STEP_ROW_ABSMAX the step requantizes as the symmetric row-wise
 * absmax INT-b baseline the paper compares against (Section 5.1): per key
 * row r'_i = max_j |X_ij| (floored at 2^-60), every c'_j = 1, and
 *   q'_ij = clip(round(X_ij q_b / r'_i), -q_b, q_b).
 * (N1 formulas.  Under N2 the levels are 2^(8-b) q: the column start and the
 * row-absmax factor divide by the top level 2^(8-b) q_b, and q_b / r' becomes
 * 2^(b-8) / r' throughout, so the largest entry still lands on +-q_b.)
 * STEPQ_STEP_ADJACENT_SLOTS is a scheduling hint, never a change of the
 * result: the tiles are then taken in launch order, which streams adjacent
 * slot records best; without it each XCD takes a contiguous run of the
 * batch, which suits scattered slots.  Set it when the batch lists adjacent
 * slots in increasing order; the results are bit-identical either way.
 * Unknown flags, or REFIT together with ROW_ABSMAX: STEPQ_E_INVALID. */
stepq_status stepq_decode_step_ex(stepq_pool *pool, const int32_t *slot_ids, int32_t batch, const void *q,
                                  const void *k, const void *v, const void *gate, const void *beta,
                                  stepq_dtype act_dtype, uint32_t flags, float *o, void *stream);

/* Memory-only reference of stepq_decode_step, a measurement aid and not
 * part of the method: one launch over the same tiles, in the same workgroup
 * order (STEPQ_STEP_ADJACENT_SLOTS as in stepq_decode_step_ex, the only flag
 * taken), moving the same memory traffic with no arithmetic.  Each tile's
 * codes (and pivot rows) are read with the decode kernels' access pattern
 * and written back unchanged, its scales are read, q, k, v, alpha and beta
 * are read (alpha as [batch][Hv]) and o is filled with zeros.  Its duration
 * is the achievable time of the step's memory pattern.  Arguments and errors
 * as stepq_decode_step; the pool's contents do not change. */
stepq_status stepq_decode_stream_ref(stepq_pool *pool, const int32_t *slot_ids, int32_t batch, const void *q,
                                     const void *k, const void *v, const void *alpha, const void *beta,
                                     stepq_dtype act_dtype, uint32_t flags, float *o, void *stream);

/* Row-impact factors w of every head (Section 4.3 and its footnote's
 * normalisation; calibrated as in Appendices A.3 and C.1), used by
 * STEPQ_STEP_REFIT.  row_weight: host [Hv][d_k] in logical row order, each
 * finite and > 0; copied.  The upload is ordered on `stream` after the
 * steps already enqueued there and before later ones, and the call returns
 * once it is done (it waits for that stream only).  Steps on other streams
 * must not be in flight on this pool.  The pool must be on the current
 * device.  A new pool has w = 1. */
stepq_status stepq_pool_set_row_weight(stepq_pool *pool, const float *row_weight, void *stream);

/* Reconstruct S^_ij = r_i c_j z_ij (Section 4.3; z the level of the code in
 * the pool's normalisation, q / q_b under N1; pivot rows: their binary16
 * values) for n slots into out [n][Hv][d_k][d_v] fp32, logical row
 * order.  Computed in fp32. */
stepq_status stepq_pool_dequant(const stepq_pool *pool, const int32_t *slot_ids, int32_t n, float *out,
                                void *stream);

/* Unpack n slots to raw codes [n][Hv][d_k][d_v] int8 (logical row order; 0
 * on pivot rows) and scales r [n][Hv][d_k] (logical order), c [n][Hv][d_v].
 * Bit-exact. */
stepq_status stepq_pool_export(const stepq_pool *pool, const int32_t *slot_ids, int32_t n, int8_t *codes,
                               float *r, float *c, void *stream);

/* Pack raw codes and scales (shapes as in stepq_pool_export) into n slots.
 * Codes must lie in [-q_b, q_b] of their row; out-of-range fields are
 * written modulo 2^b.  Bit-exact inverse of stepq_pool_export.  Pivot rows'
 * codes are ignored and their values left as they are (see
 * stepq_pool_import_pivots). */
stepq_status stepq_pool_import(stepq_pool *pool, const int32_t *slot_ids, int32_t n, const int8_t *codes,
                               const float *r, const float *c, void *stream);

/* Pivot-row values of n slots as binary16 bit patterns, pivots
 * [n][Hv][d_k][d_v] uint16 in logical row order: export writes the pivot
 * rows and zeros elsewhere; import reads the pivot rows only.  Bit-exact;
 * with stepq_pool_export / _import they save and restore a whole slot. */
stepq_status stepq_pool_export_pivots(const stepq_pool *pool, const int32_t *slot_ids, int32_t n,
                                      uint16_t *pivots, void *stream);
stepq_status stepq_pool_import_pivots(stepq_pool *pool, const int32_t *slot_ids, int32_t n,
                                      const uint16_t *pivots, void *stream);

/* Last failure message of the calling thread ("" if none). */
const char *stepq_last_error(void);

/* ---------------------------------------------------------------------------
 * CPU setup step (offline; host arrays, runs on the calling thread plus up to
 * n_threads-1 helpers; n_threads <= 0 means all hardware threads).
 */

/* Fit per-tile scales to full-precision states (Section 4.3): row factors
 *   m_i = (1/d_v) sum_j |S_ij|,   r_i = m_i^{1/2} w_i^{-1/2}
 * and absmax column factors c_j = max_i |S_ij| / r_i, so r_i c_j >= |S_ij|
 * (c is rounded upward to fp32 to keep that bound).  Both are floored at
 * 2^-60 (the positive numerical floor of Appendix C.1).  Sums in double.
 *   state [n_tiles][d_k][d_v], row_weight [n_tiles][d_k] (NULL: w = 1),
 *   r [n_tiles][d_k], c [n_tiles][d_v] (outputs). */
stepq_status stepq_setup_fit(int64_t n_tiles, int32_t d_k, int32_t d_v, const float *state,
                             const float *row_weight, float *r, float *c, int32_t n_threads);

/* stepq_setup_fit with the tiles' widths row_bits [n_tiles][d_k] (NULL: as
 * stepq_setup_fit): pivot rows (16) are left out of the column factors, as
 * the paper fits only the integer rows (Appendix C.1).  Their r entries are
 * fitted but unused. */
stepq_status stepq_setup_fit_ex(int64_t n_tiles, int32_t d_k, int32_t d_v, const float *state,
                                const float *row_weight, const uint8_t *row_bits, float *r, float *c,
                                int32_t n_threads);

/* stepq_setup_fit_ex for a pool of either level normalisation: the column
 * factors are c_j = max_i |S_ij| / (r_i top_i), top_i = 1 under N1 and
 * 2^(8-b_i) q_{b_i} under N2, so that every code of the fitted state lies in
 * [-q_b, q_b] and each column reaches the top level.  row_bits is required
 * under N2 (STEPQ_E_INVALID when NULL); levels is a stepq_levels value. */
stepq_status stepq_setup_fit_levels(int64_t n_tiles, int32_t d_k, int32_t d_v, const float *state,
                                    const float *row_weight, const uint8_t *row_bits, int32_t levels, float *r,
                                    float *c, int32_t n_threads);

/* Lifetime-aware bit allocation over key rows (Section 3.2, Eq. 6) with two
 * candidate widths lo < hi and an average budget lo <= budget <= hi.
 * gates [T][B][H] are calibration retention gates; each head's mean log
 * retention l_h = mean over (t, b) of log gates (Appendix A.3) orders its
 * rows.  With one distortion profile shared by all rows, Eq. 6 gives the wide
 * code to the floor(N (budget-lo)/(hi-lo)) rows of largest l (ties by head,
 * then row).  Output row_bits [H][d_k]. */
stepq_status stepq_setup_lifetime_bits(const double *gates, int32_t T, int32_t B, int32_t H, int32_t d_k,
                                       double budget, int32_t lo, int32_t hi, uint8_t *row_bits);

/* ---------------------------------------------------------------------------
 * Calibration side of the setup step (offline, host memory, double precision
 * sums).  Units are key rows (KDA) or whole heads (Qwen), Section 3.2.
 */

/* Row-impact factors (Section 4.3 and its footnote; Appendix A.2 with one
 * future read, Appendix C.1): per head and key row
 *   omega_i = mean_t g_{t,i}^2,  g_t = A_t^T q_t = D_t (q_t - beta_t k_t (k_t^T q_t)),
 *   w_i = omega_i^{gamma/2} / GM_j(omega_j^{gamma/2})   (the paper uses gamma = 0.25).
 * q, k [T][H][d_k], beta [T][H], gate [T][H] (gate_per_row 0: D = alpha I) or
 * [T][H][d_k] (gate_per_row 1: D = diag(d)); T calibration samples (tokens x
 * requests).  omega is floored at 2^-120.  Outputs row_weight [H][d_k] fp32
 * and, if not NULL, omega [H][d_k]. */
stepq_status stepq_setup_row_impact(int64_t T, int32_t H, int32_t d_k, const float *q, const float *k,
                                    const float *beta, const float *gate, int32_t gate_per_row, double gamma,
                                    float *row_weight, double *omega);

/* Candidate-format distortion d_u(b) (Appendix A.3): each sampled state
 * states [C][H][d_k][d_v] is coded at every candidate width b in cand_bits
 * (2, 4, 8: all non-pivot rows at b by the Key-Row-Aware Dual-Axis fit with
 * row_weight [H][d_k] (NULL: 1) -- absmax column start, one fixed-code
 * least-squares column update, a zero denominator keeping the start; 16:
 * binary16 rounding) and reconstructed.  pivots [H][d_k] (NULL: none) marks
 * rows held in binary16, left out of the column fit.
 *   unit 0 (key rows, KDA):  d_out [H*d_k][n_cand], unweighted MSE of the row;
 *   unit 1 (heads, Qwen):    d_out [H][n_cand], w_i^2-weighted MSE of the head. */
stepq_status stepq_setup_distortion(int64_t C, int32_t H, int32_t d_k, int32_t d_v, const float *states,
                                    const float *row_weight, const uint8_t *pivots, int32_t n_cand,
                                    const int32_t *cand_bits, int32_t unit, double *d_out, int32_t n_threads);

/* Lifetime weights L_u = sum_{j=0}^{horizon-1} exp(2 j ell_u) (Section 3.2)
 * from the mean log retention ell_u (Appendix A.3). */
stepq_status stepq_setup_lifetime_weights(int32_t U, const double *ell, int32_t horizon, double *L);

/* Mean log retention per unit, ell_u (Appendix A.3): the mean over the T
 * calibration samples of log g, g the gate that decays the unit's entries
 * (its own channel d_i under a channel-wise gate, gate_per_row 1, gate
 * [T][H][d_k]; its head's alpha otherwise, gate [T][H]).  unit 0 (key rows):
 * ell [H * d_k]; unit 1 (heads): ell [H], the mean over the head's rows.
 * Gates must be finite and > 0 (STEPQ_E_INVALID otherwise). */
stepq_status stepq_setup_mean_log_retention(int64_t T, int32_t H, int32_t d_k, const float *gate, int32_t gate_per_row,
                                            int32_t unit, double *ell);

/* The terms of Eq. 6's objective: cost[u][c] = L_u d_u(b_c) for the first
 * n_cand candidates of each row of d [U][d_stride] (d_stride >= n_cand). */
stepq_status stepq_setup_lifetime_costs(int32_t U, int32_t n_cand, const double *L, const double *d, int32_t d_stride,
                                        double *cost);

/* The pivot risk of Appendix C.2, the lifetime-weighted distortion an FP16
 * unit removes: risk_u = L_u (d_u(b_int) - d_u(16)), with b_int and 16 in
 * columns col_int and col_f16 of d [U][d_stride]. */
stepq_status stepq_setup_pivot_risk(int32_t U, const double *L, const double *d, int32_t d_stride, int32_t col_int,
                                    int32_t col_f16, double *risk);

/* Bit allocation (Eq. 6): choose choice[u] in [0, n_cand) minimising
 * sum_u cost[u][choice[u]] (cost = L_u d_u(b), [U][n_cand]) subject to
 * sum_u n_u b_u <= budget * sum_u n_u.
 *   method 0: multiple-choice dynamic program over spent bits (the Qwen
 *             optimizer, Appendix C.2); exact.  STEPQ_E_UNSUPPORTED when
 *             units x budget steps exceed 4e8 (use method 1).
 *   method 1: Lagrangian (the KDA optimizer): per unit argmin of
 *             cost + lam n_u b for the smallest multiplier lam that fits
 *             (bisection), then repair: repeatedly the single upgrade with
 *             the largest cost decrease per extra bit that still fits.
 * STEPQ_E_INVALID when nothing fits the budget. */
stepq_status stepq_setup_allocate(int32_t U, int32_t n_cand, const int32_t *cand_bits, const double *cost,
                                  const int32_t *n_u, double budget, int32_t method, int32_t *choice);

/* FP16 pivots (Section 3.2, Table C1): is_pivot[u] = 1 for the count units of
 * largest risk (ties: lower index), e.g. the lifetime-weighted distortion
 * reduction L_u (d_u(b) - d_u(16)) of Appendix C.2. */
stepq_status stepq_setup_select_pivots(int32_t U, const double *risk, int32_t count, uint8_t *is_pivot);

#ifdef __cplusplus
}
#endif

#endif /* STEPQ_H */
