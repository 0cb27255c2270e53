/*
 * mdgemm -- multiple-double matrix product C = A.B on one AMD Instinct MI355X (gfx950).
 *
 * Method (Chen and Verschelde, "Multiple Double Arithmetic on NVIDIA Tensor Cores"):
 * every multiple double (section 1: an unevaluated sum of nonoverlapping doubles)
 * of A is placed on one power-of-two grid shared by its row, and every element of
 * B on one grid shared by its column (section 3, balancing); its exact value is
 * then cut into S signed 13-bit integer digits (section 2, the 52-bit fraction
 * split into 13-bit quarters with exponents 0, -13, -26, -39).  Products of digits
 * need at most 26 bits, so sums of them are exact in FP64 while they stay below
 * 2^53 (section 2, the bound (NBound)).  The digit pairs (p, q) with p + q <= T are
 * multiplied as plain FP64 GEMMs on the matrix cores, pairs of one level t = p + q
 * summed together (section 2, equation (3) and the rewritten product); the levels
 * are added exactly in increasing significance and rounded into L nonoverlapping
 * limbs (section 2, steps 4-5 of the overview; section 1, renormalization).
 *
 * Conventions shared by every entry point
 *  - All array pointers are DEVICE pointers (hipMalloc, or PyTorch tensors on the
 *    GPU).  The caller allocates and owns every array.  Arrays are contiguous,
 *    limb-major (or digit/level-major), row-major planes:
 *        A [L][m][k]:  A[l*m*k + i*k + kk]      (limb 0 most significant)
 *        B [L][k][n]:  B[l*k*n + kk*n + j]
 *        C [L][m][n]:  C[l*m*n + i*n + j]
 *  - Inputs are never modified.  Outputs are fully overwritten and must not
 *    overlap any input.
 *  - Every call is asynchronous and ordered on `stream` (a hipStream_t; NULL is
 *    the default stream) unless MDGEMM_SYNC is set.  No C++ exception crosses the
 *    ABI; errors are returned as status codes.  Argument errors are detected on
 *    the host before any HIP call.
 *  - Inputs must be finite and normalized: for each element and limb l,
 *    |x[l+1]| <= ulp(x[l])/2, and x[l] == 0 implies x[l+1] == 0.  Otherwise the
 *    result is unspecified (MDGEMM_CHECK_FINITE detects non-finite limbs).
 *  - Output limbs whose magnitude falls below 2^-1022 (subnormal) are rounded by
 *    the final power-of-two scaling and are then no longer the exact greedy
 *    rounding; the products this library is built for stay far from that range.
 *    Zero limbs, including limbs that underflow to zero, are +0.0.
 */
#ifndef MDGEMM_H
#define MDGEMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------------- */
#define MDGEMM_OK 0
#define MDGEMM_EINVAL -1      /* invalid size, limb/slice/cutoff count, null or overlapping pointer */
#define MDGEMM_EEXACT -2      /* pairs_t * k * (2^w - 1)^2 >= 2^53 (2^31 with MDGEMM_INT8) for a kept level t */
#define MDGEMM_ENOMEM -3      /* the library's own workspace could not be allocated */
#define MDGEMM_EHIP -4        /* a HIP call failed (no device, launch or runtime error) */
#define MDGEMM_EWORKSPACE -5  /* the caller's workspace is smaller than mdgemm_workspace_bytes() */
#define MDGEMM_ENONFINITE -6  /* MDGEMM_CHECK_FINITE: an input limb is inf or nan */

/* ---- limits ---------------------------------------------------------------- */
#define MDGEMM_MAX_LIMBS 16   /* double (1), double-double (2), ... quad (4), octo (8), hexa double (16) */
#define MDGEMM_MAX_SLICES 68  /* digits per element */
#define MDGEMM_MAX_LEVELS 135 /* 2 * MDGEMM_MAX_SLICES - 1 */
#define MDGEMM_SLICE_BITS 13      /* digit width of section 2 */
#define MDGEMM_MAX_SLICE_BITS 26  /* widest digit: a product of two stays below 2^52 */
#define MDGEMM_MAX_DIGIT_BITS 908 /* slices * slice_bits + 52 <= 15 64-bit words */
#define MDGEMM_Z_WORDS 28         /* 64-bit words per element written by mdgemm_accumulate */

/* slice_bits selector for mdgemm_opts.slice_bits (else an explicit width 1..26) */
#define MDGEMM_SLICE_BITS_AUTO -1 /* the width with the fewest pairs that stays exact for this k */

/* ---- flags for mdgemm_opts.flags ------------------------------------------- */
#define MDGEMM_CHECK_FINITE 1u /* scan A and B for inf/nan first; synchronizes the stream */
#define MDGEMM_SYNC 2u         /* synchronize the stream before returning and report kernel errors */
#define MDGEMM_TIME_STAGES 4u  /* record HIP events between stages; read with mdgemm_stage_times() */
#define MDGEMM_KARATSUBA 8u    /* level products by the Karatsuba schedule where it pays (see below) */
#define MDGEMM_KARATSUBA_MIN_TERMS 16u /* the Karatsuba schedule with the fewest GEMMs, always */
#define MDGEMM_INT8 32u        /* level products on the int8 matrix cores, digits of at most 7 bits (see below) */
#define MDGEMM_STAGED 64u      /* always the staged kernels, never the fused small-product kernel (see below) */
#define MDGEMM_GROUP_SIGN 128u      /* section 3's sign groups: A = A+ + A-, B likewise, four products (see below) */
#define MDGEMM_GROUP_EXPONENT 256u  /* section 3's exponent classes over range_bits (see below) */

/* cutoff selectors for mdgemm_opts.cutoff (else an explicit T in 0 .. 2S-2) */
#define MDGEMM_CUTOFF_DEFAULT -1  /* T = S - 1: the pair set of the rewritten product */
#define MDGEMM_CUTOFF_ALL -2      /* T = 2S - 2: every slice pair */

typedef struct mdgemm_opts {
  void* stream;           /* hipStream_t to launch on; NULL = default stream */
  void* workspace;        /* caller-owned device buffer; NULL = library-owned buffer (see below) */
  size_t workspace_bytes; /* size of `workspace` in bytes */
  int slices_per_limb;    /* 13-bit digits per limb, S = limbs * slices_per_limb; 0 = the default count (below) */
  int cutoff;             /* largest kept p + q; MDGEMM_CUTOFF_DEFAULT or _ALL or 0..2S-2 */
  unsigned flags;         /* MDGEMM_CHECK_FINITE, _SYNC, _TIME_STAGES, _KARATSUBA, _KARATSUBA_MIN_TERMS, _INT8,
                             _STAGED, _GROUP_SIGN, _GROUP_EXPONENT */
  int slice_bits;         /* digit width w: 0 = 13 (section 2), 1..26, or MDGEMM_SLICE_BITS_AUTO */
  int slices;             /* digits per element S; 0 = derived (see below) */
  int range_bits;         /* range balancing: full precision down to 2^-range_bits of the line; 0 = off */
} mdgemm_opts;

/* Workspace.  A caller workspace is used by this call only; calls that share one
 * must be ordered by the caller.  Without one, the library keeps one buffer per
 * device, grown on demand: calls that use it are ordered among themselves on the
 * GPU (each waits for the previous user's work, across streams), and such a call
 * is refused with MDGEMM_EINVAL while its stream is capturing a graph (the graph
 * would keep an address that a later, larger call may free). */

/* Digit width and count.
 *  - The default count of 13-bit digits, S13(L): four per limb up to quad
 *    doubles (section 2's quarters, 52 L bits, which cover the 53 L - 4 bits of
 *    the tolerance 4 k 2^-(53 L - 4) (|A||B|)); for five or more limbs, where four
 *    per limb fall short of those bits, ceil((53 L - 4) / 13) + 1 (one guard digit
 *    for the levels dropped at T = S - 1): 34 for octo and 66 for hexa doubles.
 *  - slice_bits 0 or 13: w = 13 and S = slices, else limbs * slices_per_limb,
 *    else (slices_per_limb 0) S13(L).
 *  - slice_bits 1..26 (the adaptive width, wider digits and fewer of them): S =
 *    slices, else ceil(13 S13(L) / w), at least the digit bits of the default.
 *  - MDGEMM_SLICE_BITS_AUTO (slices must be 0): among w = 13..26 with
 *    S = ceil(13 S13(L) / w) and the requested cutoff (T = S - 1 by default), those
 *    whose levels stay exact (max pairs of a level times k (2^w - 1)^2 < 2^53), the
 *    one with the fewest pairs, the wider on a tie; MDGEMM_EEXACT when none
 *    qualifies.  Double-double at k = 4096 gets w = 19,
 *    S = 6 (21 pairs instead of 36); the digits cover at least as many bits as
 *    the default 13-bit digits, so the product is at least as accurate.
 * Range balancing (section 3, grouping by exponent so that smaller numbers keep
 * their bits): with range_bits > 0 every line keeps its one grid and gets
 * D = ceil(range_bits / w) more digits, S = S0 + D where S0 is the count above,
 * and the default cutoff becomes T = S0 - 1 + 2D.  An element whose exponent is
 * at most range_bits below its line's exponent then keeps S0 digits of its own,
 * and the product of two such elements keeps its levels down to S0 - 1 below
 * its own leading level.  With MDGEMM_SLICE_BITS_AUTO the width is chosen for the
 * fewest pairs of (S, T) including D.  mdgemm_line_spread measures the range of
 * the data.
 * In every case S <= MDGEMM_MAX_SLICES and S w <= MDGEMM_MAX_DIGIT_BITS; the Karatsuba
 * schedules combine at most 64 digits (products with more keep the pair schedule).
 *
 * MDGEMM_INT8.  The level sums of section 2 are exact integer sums, so with
 * digits of at most 7 bits (|d| <= 127) they are formed on the int8 matrix cores
 * with exact int32 sums over the contiguous digit ranges of each level's pairs,
 * which requires max pairs of a level times k (2^w - 1)^2 < 2^31.  slice_bits 0
 * or MDGEMM_SLICE_BITS_AUTO: the widest w <= 7 whose levels stay exact for this k,
 * S = ceil(13 S13(L) / w) (plus the range digits), T by the cutoff rules above
 * (T = S - 1 by default); slice_bits 1..7: that width; wider, the Karatsuba flags,
 * or S > 64 (more than 8 limbs at w = 7) return MDGEMM_EINVAL, and no exact width
 * MDGEMM_EEXACT.  Digits, levels and C are bit-identical to the FP64 path run
 * with the same slice_bits, slices and cutoff.  Double-double at k = 4096:
 * w = 7, S = 15, T = 14 (120 pairs).  The level products run on the library's
 * own int8 kernel, all levels in one launch. */

/* Grouped products (section 3, the balancing problems: numbers grouped by sign,
 * A = A+ + A-, and by the exponent of their leading part, A = A_0 + A_1 + ...,
 * each group multiplied with each group of the other operand).
 *  - MDGEMM_GROUP_EXPONENT: every line keeps its grid exponent E; an element
 *    whose leading limb has frexp exponent e is in class
 *    c = min(Ge - 1, floor((E - e) / w)), with Ge = 1 + ceil(range_bits / w)
 *    classes, and its digits are taken on the class grid E - c w (so it keeps
 *    its leading bits); range_bits then sets the classes instead of adding
 *    digits: S = S0 + 1 (the element lies up to one digit below its class
 *    grid) and the default cutoff T = S0 + 1 (S0 the digit count without range
 *    balancing), applied to every class pair.
 *  - MDGEMM_GROUP_SIGN: positive and negative elements in separate groups on the
 *    same grid (both flags: 2 Ge groups).
 * Every group pair (g, h) contributes its pairs p + q <= T at level
 * p + q + c(g) + c(h), so the product has T + 1 + 2 (Ge - 1) levels, and every
 * element belongs to one group, so a level's sums keep the bound of the pair
 * schedule (pairs_t k (2^w - 1)^2 < 2^53 over the pairs of one group pair).
 * mdgemm_plan reports S (digits per group) and T (per group pair).  Sign groups
 * give the same digits summed in a different grouping: the limbs equal the
 * ungrouped product's bit for bit, at four times the pairs.  Up to 4 limbs and
 * w S + 52 <= 384; not with MDGEMM_INT8, the Karatsuba flags or
 * MDGEMM_SLICE_BITS_AUTO (MDGEMM_EINVAL).  The workspace holds G S digit panels
 * of each operand and the T + 1 + 2 (Ge - 1) level planes. */

/* Small products.  For an output of at most 256 tiles of 16 x 16 (up to 4
 * limbs, digits of at most 24 bits, at most 32 levels, the level sum of an
 * element within 448 bits and the split's integer within 320 bits), whose
 * estimated time is below the staged path's (estimates fitted to products of 1
 * to 4 limbs measured both ways on MI355X; the fused time grows with k (S + L)
 * and with the level products of the most loaded SIMD, the staged time with its
 * level GEMM's heaviest block), mdgemm_ex runs all five steps in one launch of a
 * fused kernel per 16 x 16 tile of C instead of the staged kernels: the same
 * digits, levels and limbs bit for bit, without launches in between and
 * without the workspace (a caller workspace is still checked but not written;
 * the library buffer is not used, so such calls can be captured in a HIP graph
 * without a workspace).  Not with MDGEMM_INT8, the Karatsuba flags or
 * MDGEMM_CHECK_FINITE; MDGEMM_STAGED turns it off.  With MDGEMM_TIME_STAGES the
 * whole kernel counts as the level-product stage. */

/* Logging.  With the environment variable MDGEMM_LOG=1 (read once per process)
 * every call of mdgemm, mdgemm_ex, mdgemm_ex_noalloc and mdgemm_qr_dd writes one
 * line to stderr when it returns: its sizes, the plan (w, S, T; "unplanned" for
 * arguments that do not resolve), the flags, the workspace kind, the stream, the
 * path taken (refused, empty, zero (k = 0), fused small product, staged: pair
 * levels / karatsuba / grouped products, int8 levels) and the status string.
 * MDGEMM_LOG=2 also logs the products a QR makes.  Unset or 0: silent. */

/* Fill `opts` with the defaults: default stream, library workspace, the default
 * count S13(L) of 13-bit digits (slices_per_limb 0), cutoff T = S - 1, no range
 * balancing, no flags. */
void mdgemm_opts_init(mdgemm_opts* opts);

/* The digit width, digit count and cutoff mdgemm_ex uses for this product and
 * these options (opts may be NULL), written to *slice_bits, *slices, *cutoff
 * (each pointer may be NULL).  Returns MDGEMM_OK, MDGEMM_EINVAL or MDGEMM_EEXACT. */
int mdgemm_plan(int64_t m, int64_t n, int64_t k, int limbs, const mdgemm_opts* opts, int* slice_bits, int* slices,
                int* cutoff);

/* C = A.B for L-limb operands (L = limbs in 1..16) with the default options (the
 * default count S13(L) of 13-bit digits, T = S - 1).
 * m, n, k >= 0; m == 0 or n == 0 does nothing; k == 0 writes C = +0.0; m and n at
 * most 2^27 (MDGEMM_EINVAL beyond).
 * Returns MDGEMM_OK or a negative status. */
int mdgemm(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C);

/* Bytes of device workspace mdgemm_ex needs for this product and these options
 * (0 for an empty product; SIZE_MAX for invalid arguments).  Layout, each part
 * aligned to 256 bytes: EA int32[m], EB int32[n], flag int32, the schedule's
 * job table (32-bit words), the combination panels of A [CA][kp][mp] and of
 * B [CB][kp][np] (FP32 with kp = k rounded up to 32 when every panel value is
 * below 2^24 (mdgemm_schedule_info, info[10]), else FP64 with kp = k rounded up
 * to 16; mp and np = m and n rounded up to 128; the first S combinations are the
 * digits, CA = CB = S for the pair schedule), the GEMM output planes f64[P][m][n]
 * (P = T+1 levels for the pair schedule, the schedule's planes for
 * MDGEMM_KARATSUBA).  With MDGEMM_INT8: EA, EB, flag, A's int8 digits
 * [mp][128 + S kp] and B's [np][128 + S kp] (rows of 128 zero bytes and the S
 * digits' k ranges; kp = k rounded up to 128, mp and np = m and n rounded up
 * to 256), the int32 level planes [T+1][m][n]. */
size_t mdgemm_workspace_bytes(int64_t m, int64_t n, int64_t k, int limbs, const mdgemm_opts* opts);

#define MDGEMM_LAYOUT_INFO 12 /* entries written by mdgemm_workspace_layout */

/* Where mdgemm_ex keeps each stage's output inside a caller workspace, for
 * checking a product's intermediate results (the workspace is not cleared
 * after the call, so after mdgemm_ex returns and its stream is synchronized
 * the parts hold that call's exponents, digits and level products).  Host
 * only.  Writes min(count, MDGEMM_LAYOUT_INFO) values:
 *   info[0] byte offset of EA int32[m],   info[1] of EB int32[n],
 *   info[2] of A's digit panels [CA][kp][mp] (A transposed: [s][kk][i] = digit s
 *     of A[i][kk]), info[3] of B's digit panels [CB][kp][np] ([s][kk][j] = digit
 *     s of B[kk][j]); the first S panels are the digits, zero padded,
 *   info[4] of the output planes f64 [P][m][n] (the levels G_t, t = 0..T, when
 *     info[10] == 1),
 *   info[5] bytes per panel value (4: FP32, 8: FP64), info[6] kp, info[7] mp,
 *   info[8] np, info[9] P, info[10] 1 for the pair schedule (planes = levels),
 *   info[11] mdgemm_workspace_bytes().
 * Returns the count written, MDGEMM_EEXACT, or MDGEMM_EINVAL (also for an empty
 * product, with MDGEMM_INT8, whose layout is not described here, and for a
 * product that runs the fused small-product kernel, which leaves nothing in the
 * workspace; MDGEMM_STAGED selects the staged kernels). */
int mdgemm_workspace_layout(int64_t m, int64_t n, int64_t k, int limbs, const mdgemm_opts* opts, int64_t* info,
                            int count);

/* C = A.B with explicit options (opts may be NULL for the defaults).  Runs, in
 * stream order: row exponents of A and column exponents of B, the splits of A
 * and B into digits, the level GEMMs, and the exact accumulation and rounding
 * into C.  With a caller workspace smaller than mdgemm_workspace_bytes() it
 * returns MDGEMM_EWORKSPACE, and with one that overlaps A, B or C it returns
 * MDGEMM_EINVAL; in both cases it launches nothing. */
int mdgemm_ex(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C,
              const mdgemm_opts* opts);

/* ---- allocation-free entry point ---------------------------------------------
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): mdgemm_ex on a fixed
 * device scratch array of MDGEMM_NOALLOC_MAX_BYTES bytes that the library holds,
 * one per device it runs on, from when the library is loaded on that device
 * until the process ends.  The caller passes A, B and C as for mdgemm_ex and
 * opts with no workspace (workspace NULL, workspace_bytes 0); MDGEMM_TIME_STAGES
 * and MDGEMM_CHECK_FINITE are refused (MDGEMM_EINVAL).  A product whose
 * mdgemm_workspace_bytes() exceeds MDGEMM_NOALLOC_MAX_BYTES returns
 * MDGEMM_EWORKSPACE and launches nothing.  The call allocates no device memory
 * (no hipMalloc, hipFree or allocating library routine).  Every call on one
 * device shares that device's scratch array, which keeps the last call's
 * contents: calls that may overlap in time on one device (other streams, other
 * host threads) race and must be ordered by the caller.  Results equal
 * mdgemm_ex's bit for bit. */
#define MDGEMM_NOALLOC_MAX_BYTES 67108864 /* 64 MiB of scratch per device */

int mdgemm_ex_noalloc(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C,
                      const mdgemm_opts* opts);

/* Milliseconds spent in each stage of the last mdgemm_ex call that set
 * MDGEMM_TIME_STAGES on this process: ms[0] exponents, ms[1] splits,
 * ms[2] level GEMMs, ms[3] accumulation and rounding.  Waits for that call's
 * last event.  Writes min(count, 4) values and returns how many, or a negative
 * status.  Not meant for concurrent timed calls from several threads. */
int mdgemm_stage_times(float* ms, int count);

/* Static text for a status code. */
const char* mdgemm_status_string(int status);

/* Free the library-owned workspace of every device (after synchronizing them). */
void mdgemm_release(void);

/* ---- stage entry points (the same kernels as mdgemm_ex) --------------------- */

/* Step a1, balancing (section 3; per-line grid after the worked example of
 * section 2).  X0 is the leading-limb plane [rows][cols].  axis 0: E[i] for every
 * row i (E has `rows` entries); axis 1: E[j] for every column j (`cols` entries).
 * E = the largest frexp exponent (x = f 2^E, 1/2 <= |f| < 1) of a nonzero entry of
 * the line; 0 for an all-zero line.  Subnormals get their true exponent. */
int mdgemm_exponents(int64_t rows, int64_t cols, int axis, const double* X0, int32_t* E, void* stream);

/* The exponent range of every line, for choosing mdgemm_opts.range_bits (section
 * 3: the exponents a group of numbers spans).  E as mdgemm_exponents; spread[line]
 * = E[line] - the smallest frexp exponent of a nonzero entry of the line, 0 for an
 * all-zero line.  E and spread have `rows` (axis 0) or `cols` (axis 1) entries
 * and must not overlap. */
int mdgemm_line_spread(int64_t rows, int64_t cols, int axis, const double* X0, int32_t* E, int32_t* spread,
                       void* stream);

/* Step a2, the exact split (section 2 worked example; sections 2-3 balancing and
 * the opposite-sign transfer).  X [limbs][rows][cols], E from mdgemm_exponents
 * with the same axis, D [slices][rows][cols] (float64, integer valued).  For each
 * element with exact value V on grid exponent E and digit width w = slice_bits
 * (13 in section 2): D_abs = floor(|V| / 2^(E - w S)),
 * digit s = sign(V) * bits w(S-1-s) .. w(S-s)-1 of D_abs, so that
 * V = sum_s digit_s 2^(E - w(s+1)) + R with |R| < 2^(E - w S) and R V >= 0.
 * Zero digits are +0.0.  Requires |V| < 2^E (true for normalized input and the
 * exponents of mdgemm_exponents).  limbs 1..16, slices 1..64, slice_bits 1..26,
 * slices * slice_bits <= 844. */
int mdgemm_split(int64_t rows, int64_t cols, int limbs, int slices, int slice_bits, int axis, const double* X,
                 const int32_t* E, double* D, void* stream);

/* Step a2 into the operand layout of mdgemm_slice_gemm ("panels"): the same
 * digits as mdgemm_split, k-major and zero-padded to whole GEMM tiles, with
 * kp = cols rounded up to 16 for axis 0 (rows up to 16 for axis 1) and
 * cp = rows (axis 0) or cols (axis 1) rounded up to 128:
 *   axis 0 (A, rows = m, cols = k):  D [slices][kp][cp], D[s][kk][i] = digit s of A[i][kk];
 *   axis 1 (B, rows = k, cols = n):  D [slices][kp][cp], D[s][kk][j] = digit s of B[kk][j].
 * Every padding entry is +0.0.  Arguments and requirements as mdgemm_split. */
int mdgemm_split_panel(int64_t rows, int64_t cols, int limbs, int slices, int slice_bits, int axis,
                       const double* X, const int32_t* E, double* D, void* stream);

/* Step a3, the slice GEMMs (section 2, equation (3) and the rewritten product).
 * DAt and DBp are digit panels (see mdgemm_split_panel) with |digit| <= 2^w - 1,
 * w = slice_bits (8191 for the 13-bit digits of section 2):
 * DAt [S][kp][mp] holds A's digits transposed, DBp [S][kp][np] holds B's, where
 * kp = k rounded up to 16, mp = m and np = n rounded up to 128, zero padding;
 * both pointers 16-byte aligned.
 * per_pair == 0: out [T+1][m][n], out[t] = sum over p + q = t (0 <= p, q < S) of
 * DA_p . DB_q for t = 0..cutoff.  per_pair != 0: out [S][S][m][n],
 * out[p][q] = DA_p . DB_q for every p + q <= cutoff (other planes untouched; one
 * launch).
 * Exact in FP64 (any summation order) because every partial sum is an integer
 * below 2^53; returns MDGEMM_EEXACT when pairs_t * k * (2^w - 1)^2 >= 2^53.
 * S in 1..64, slice_bits 1..26, cutoff in 0..2S-2. */
int mdgemm_slice_gemm(int64_t m, int64_t n, int64_t k, int slices, int slice_bits, int cutoff, int per_pair,
                      const double* DAt, const double* DBp, double* out, void* stream);
/* (The job table of mdgemm_slice_gemm is placed in the library buffer, so the
 * call is refused with MDGEMM_EINVAL while `stream` captures a graph.) */

/* ---- schedules of the level products ----------------------------------------
 * Section 2 (equation (3), the rewritten product) multiplies every digit pair
 * (p, q) with p + q <= T and sums the pairs of a level t = p + q: the pair
 * schedule, (T+1) levels from sum_t pairs_t GEMMs of length k.  With the digits
 * of an element read as the coefficients of a polynomial in 2^-w, level t is
 * coefficient t of the product of two polynomials, and Karatsuba's identity
 * (a0 + a1 x)(b0 + b1 x) = a0 b0 + x [(a0 + a1)(b0 + b1) - a0 b0 - a1 b1] + x^2 a1 b1,
 * applied recursively and truncated at T, forms the same coefficients from
 * fewer products of digit sums ("combinations").  Everything stays integer:
 * combinations are exact, every GEMM job keeps k * sum(|comb a| |comb b|) *
 * (2^w - 1)^2 < 2^53 (|comb| = digits in the sum), and the levels are formed
 * from the planes in 64-bit integers, so both schedules give bit-identical
 * levels and products.  Double-double with T = 7 takes 24 products instead of
 * 36, quad-double (16 digits, T = 15) 69 instead of 136.  The schedule also
 * costs output planes (one per distinct set of level coefficients), level
 * entries in the accumulation and combination panels; the planner weighs them
 * against the GEMMs for the product's shape (m, n, k) with rates measured on
 * MI355X and keeps the pair schedule where Karatsuba would not pay (small
 * products, whose combination panels cost as much as a GEMM).
 * MDGEMM_KARATSUBA_MIN_TERMS takes the plan with the fewest GEMMs whatever the
 * other costs (it overrides MDGEMM_KARATSUBA). */

#define MDGEMM_SCHEDULE_INFO 12 /* entries written by mdgemm_schedule_info */

/* Size of the schedule mdgemm_ex uses for an m x k by k x n product with
 * S = slices digits of slice_bits bits, cutoff T, and flags (MDGEMM_KARATSUBA,
 * MDGEMM_KARATSUBA_MIN_TERMS, or 0 for the pair schedule).  Writes min(count, MDGEMM_SCHEDULE_INFO) values:
 *   info[0] GEMM terms (products of two combinations, k long each),
 *   info[1] GEMM jobs, info[2] output planes, info[3] combinations of A,
 *   info[4] combinations of B, info[5] level entries, info[6] largest job weight
 *   sum(|comb a| |comb b|), info[7] deepest combination (0 = digits only),
 *   info[8] 1 when the planes are the levels themselves (pair schedule),
 *   info[9] digits in the largest combination (1 for the pair schedule),
 *   info[10] 1 when mdgemm_ex keeps the panels in FP32 (every panel value, at
 *     most info[9] (2^w - 1), below 2^24: exact; k rounded up to 32), else FP64,
 *   info[11] k chunks per job: products whose tile jobs would not fill the GPU
 *     split k into up to 8 chunks, each writing its own plane (the planes of a
 *     job's chunks enter the same levels; partial sums of integers, exact).
 * Host only (no HIP call).  Returns the count written or MDGEMM_EINVAL. */
int mdgemm_schedule_info(int64_t m, int64_t n, int64_t k, int slices, int slice_bits, int cutoff, unsigned flags,
                         int64_t* info, int count);

/* The schedule itself, for checking (host only).  Any pointer may be NULL;
 * sizes from mdgemm_schedule_info:
 *   mask_a[CA], mask_b[CB]: the digit set of every combination (bit p = digit p);
 *   parents_a[2 CA], parents_b[2 CB]: combination c >= S is the sum of
 *     combinations parents[2c] and parents[2c+1] (-1, -1 for the digits c < S);
 *   jobs[4 J]: first pair, pair count, output plane and k chunk (0 .. info[11]-1,
 *     a 1/info[11] share of the k steps of every pair) of job j;
 *   pairs[2 terms]: (combination of A, combination of B) of every pair;
 *   plane_first[P + 1], entries[2 E]: plane j enters the levels
 *     entries[2e] with coefficient entries[2e+1] for plane_first[j] <= e < plane_first[j+1].
 * Returns MDGEMM_OK or MDGEMM_EINVAL. */
int mdgemm_schedule_export(int64_t m, int64_t n, int64_t k, int slices, int slice_bits, int cutoff, unsigned flags,
                           uint64_t* mask_a, int32_t* parents_a, uint64_t* mask_b, int32_t* parents_b, int32_t* jobs,
                           int32_t* pairs, int32_t* plane_first, int32_t* entries);

/* Workspace bytes of mdgemm_schedule_levels (SIZE_MAX for invalid arguments). */
size_t mdgemm_schedule_workspace_bytes(int64_t m, int64_t n, int64_t k, int slices, int slice_bits, int cutoff,
                                       unsigned flags);

/* Step a3 by a schedule: the levels G [cutoff+1][m][n] (integer-valued doubles)
 * of the digit panels DAt [S][kp][mp] and DBp [S][kp][np] (as for
 * mdgemm_slice_gemm), computed by the schedule that `flags` selects
 * (MDGEMM_KARATSUBA or 0): the digit panels are copied into the workspace, the
 * combinations formed, the schedule's GEMMs run, and for the Karatsuba schedule
 * the levels formed from the planes in 64-bit integers.  The result equals
 * mdgemm_slice_gemm(per_pair = 0) bit for bit.  workspace: caller-owned device
 * buffer of mdgemm_schedule_workspace_bytes() bytes, or NULL for the library
 * buffer (then refused with MDGEMM_EINVAL while `stream` captures a graph).
 * Returns MDGEMM_EEXACT when pairs_t * k * (2^w - 1)^2 >= 2^53. */
int mdgemm_schedule_levels(int64_t m, int64_t n, int64_t k, int slices, int slice_bits, int cutoff, unsigned flags,
                           const double* DAt, const double* DBp, double* G, void* workspace, size_t workspace_bytes,
                           void* stream);

/* Step a4 alone, the exact accumulation (section 2, steps 4-5), exported for
 * checking.  G [levels][m][n] integer-valued with |G| < 2^53, levels 1..127,
 * w = slice_bits 1..26 with w (levels - 1) + 55 <= 1792 (the sum fits 28 words).  Writes the integer
 * N = sum_t G_t 2^(w (levels-1-t)) as MDGEMM_Z_WORDS 64-bit two's-complement
 * words, least significant first: Z [MDGEMM_Z_WORDS][m][n] int64.  The
 * accumulated value is N 2^(-w (levels-1)) (before the grid scale). */
int mdgemm_accumulate(int64_t m, int64_t n, int levels, int slice_bits, const double* G, int64_t* Z, void* stream);

/* Steps a4 + a5: exact accumulation of the levels and rounding into `limbs`
 * nonoverlapping doubles (section 1, renormalization; section 2, adding the parts
 * into a multiple double), times the grid scale 2^(EA[i] + EB[j] - 2w),
 * w = slice_bits (13: 2^(EA + EB - 26)):
 * with Z = sum_t G_t 2^(-w t), C[.][i][j] = (c_0, .., c_{L-1}) 2^(EA[i]+EB[j]-2w)
 * where c_0 = RN(Z) and c_l = RN(Z - c_0 - .. - c_{l-1}) (round to nearest, ties
 * to even).  G [levels][m][n] (levels 1..127, w (levels - 1) + 55 <= 1792), EA int32[m],
 * EB int32[n], C [limbs][m][n] (limbs 1..16). */
int mdgemm_accum_renorm(int64_t m, int64_t n, int limbs, int levels, int slice_bits, const double* G,
                        const int32_t* EA, const int32_t* EB, double* C, void* stream);

/* ---- application: blocked Householder QR in double-double --------------------
 * The downstream use the paper names as future work (section 5): A = Q R for a
 * double-double matrix, with the trailing updates of each panel on mdgemm_ex. */

/* Workspace bytes of mdgemm_qr_dd (SIZE_MAX for invalid arguments: m >= n >= 1,
 * nb in 1..64, m and n at most 2^20). */
size_t mdgemm_qr_dd_workspace_bytes(int64_t m, int64_t n, int nb);

/* Householder QR of A [2][m][n] (double-double, limb-major, m >= n), in place:
 * A = Q R with Q = H_0 ... H_{n-1}, H_j = I - tau_j v_j v_j^T, v_j(j) = 1 and
 * v_j zero above row j.  On return A holds R on and above the diagonal (R(j, j)
 * >= 0) and v_j below it (LAPACK's convention), tau [2][n] the tau_j (all in
 * double-double).  Panels of nb columns (1..64) are factored in double-double
 * arithmetic (Golub and Van Loan's Householder vector) by workgroups of 8 rows
 * (panels of at most 1024 rows), 16 (at most 2048) or 32, one launch per column,
 * a single reduction serving both the column's norm and the reflection's dot
 * products;
 * each panel's reflections are accumulated as I - V T V^T (T upper triangular)
 * and the columns to its right updated as A2 - V (T^T (V^T A2)), three products
 * on mdgemm_ex at the adaptive digit width.  workspace: caller-owned device buffer of
 * mdgemm_qr_dd_workspace_bytes() bytes, not overlapping A or tau.  Stream
 * ordered; returns MDGEMM_OK, MDGEMM_EINVAL, MDGEMM_EWORKSPACE or a status of
 * mdgemm_ex.  Inputs must be finite and normalized double-doubles. */
int mdgemm_qr_dd(int64_t m, int64_t n, int nb, double* A, double* tau, void* workspace, size_t workspace_bytes,
                 void* stream);

/* ---- application: Taylor series of the solution of a power-series system ----
 * The application the paper names for the QR (section 5): the coefficients of
 * X(t) = X_0 + X_1 t + ... + X_d t^d with A(t) X(t) = B(t) modulo t^(d+1). */

/* Workspace bytes of mdgemm_taylor_dd (SIZE_MAX for invalid arguments: n in
 * 1..32768, r in 1..2^20, d in 0..1024). */
size_t mdgemm_taylor_dd_workspace_bytes(int64_t n, int64_t r, int d);

/* Solve A(t) X(t) = B(t) modulo t^(d+1) for matrix power series in
 * double-double: A [d+1][2][n][n] holds A_0 .. A_d, B [d+1][2][n][r] holds
 * B_0 .. B_d, X [d+1][2][n][r] receives X_0 .. X_d (each coefficient a limb-major
 * double-double block), such that A_0 X_k = B_k - sum_{i=1..k} A_i X_{k-i}.
 * A_0 must be nonsingular (a singular or numerically singular A_0 leaves
 * non-finite or meaningless values in X; no check is made).  Method: the QR of
 * A_0 (as mdgemm_qr_dd, 64-column panels) with its reflections applied to an
 * identity block, which gives Q^T; blocked back substitution with R turns it
 * into M = R^-1 Q^T; then for each degree X_k = M (B_k - [A_k ... A_1]
 * [X_0; ...; X_{k-1}]), two products on mdgemm_ex at the adaptive digit width.
 * workspace: caller-owned device buffer of mdgemm_taylor_dd_workspace_bytes()
 * bytes, overlapping none of A, B and X; X overlaps neither A nor B.  Stream
 * ordered; returns MDGEMM_OK, MDGEMM_EINVAL, MDGEMM_EWORKSPACE or a status of
 * mdgemm_ex.  Inputs must be finite and normalized double-doubles. */
int mdgemm_taylor_dd(int64_t n, int64_t r, int d, const double* A, const double* B, double* X, void* workspace,
                     size_t workspace_bytes, void* stream);

/* ---- calibration (measurement aids, not part of the product) ---------------
 * The rates the stages are measured against, on the caller's device. */

/* Launches `blocks` workgroups of 256 threads that each run `iters` rounds of
 * eight independent v_mfma_f64_16x16x4f64 per wave (no memory traffic in the
 * loop) and write one double per thread to sink [blocks * 256] (device memory).
 * Time it with events on `stream` to measure the sustainable FP64 MFMA rate.
 * Returns the FP64 flops the launch performs (2 * 16 * 16 * 4 per instruction),
 * or a negative status (blocks in 1 .. 2^24, iters >= 1). */
int64_t mdgemm_probe_mfma_f64(int64_t blocks, int64_t iters, double* sink, void* stream);

/* dst[0 .. count) = src[0 .. count) with 32-byte vector loads and stores
 * (count a multiple of 4, both pointers 32-byte aligned, not overlapping):
 * reads and writes 8 count bytes each, the HBM rate of a plain stream. */
int mdgemm_probe_copy(const double* src, double* dst, int64_t count, void* stream);

/* Plain streaming rate for a read/write mix: out of src [reads][count] (doubles,
 * plane stride count) every element's planes are read and [writes][count]
 * doubles written to dst.  reads 1..256, writes 0..256; the two regions must not
 * overlap.  Stream ordered; returns MDGEMM_OK, MDGEMM_EINVAL or MDGEMM_EHIP.
 * bench.py times it at the size and mix of the exponent, split and
 * accumulation stages. */
int mdgemm_probe_stream(const double* src, int reads, double* dst, int writes, int64_t count, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MDGEMM_H */
