/*
 * fabft.h - C ABI of the Flash-ABFT attention forward library (libfabft.so)
 * for AMD Instinct MI355X (gfx950).
 *
 * Flash-ABFT (arXiv 2507.16676) computes attention O = softmax(scale*Q K^T) V
 * (Eq. 1) with the one-pass FlashAttention-2 recurrence and, fused into the
 * same pass, a predicted output checksum per query row (Algorithm 3):
 *
 *   c <- c * exp(m_old - m_new) + sumrow_k(V) * exp(s_k - m_new)
 *
 * where sumrow_k(V) is the sum of row k of V (Eq. 4). After the last key
 * block, pred = c / l is the predicted sum of the output row (Eq. 8) and is
 * compared with the actual row sum of O: one check per query row.
 *
 * Conventions for every entry point:
 *  - q, k, v, o are DEVICE pointers to bfloat16 bit patterns (uint16),
 *    contiguous row-major [B, H, Lq, d] (q, o) and [B, H, Lk, d] (k, v),
 *    16-byte aligned. resid is fp32 [B, H, Lq], flags is uint8 [B, H, Lq],
 *    pred/actual (when given) fp32 [B, H, Lq]; all device pointers.
 *  - The caller owns every buffer. The library allocates nothing (one entry
 *    point uses a static device array of its own instead of a workspace) and
 *    keeps only a stream, the detection thresholds, the weighted- and
 *    score-check switches and the launch shape as process-global state
 *    (setters are not thread-safe).
 *  - d must be 64, 96, 128 or 256 (d = 96 runs the d = 128 kernels with the
 *    columns 96..127 zero on chip: identical results, 4/3 of the work).
 *    B, H, Lq, Lk >= 1. scale must be finite and >= 0; a scale below
 *    2^-126 / log2(e) (zero included) runs as that value, which weighs every
 *    visible key alike for scores below 2^100 in magnitude.
 *  - causal != 0 keeps key k for query i iff k <= i + (Lk - Lq)
 *    (bottom-right aligned; the plain lower triangle when Lq == Lk). A query
 *    row with no visible key gets O = 0, pred = actual = resid = 0, flag 0.
 *  - Arguments are validated before anything is launched; on error a
 *    negative status is returned and nothing is written. Launches are
 *    asynchronous on the library stream; FABFT_E_LAUNCH reports a launch
 *    failure seen by hipGetLastError; device faults surface at the caller's
 *    next synchronisation. Production entry points never synchronise.
 *  - Computation: bf16 MFMA with fp32 accumulation for Q K^T and P V; the
 *    softmax weights fed to P V are rounded to bf16 (p~), and the checksum
 *    uses exactly those p~; l, c, the row sums and the residual are fp32.
 *    (The key split with at most four query rows computes both products on
 *    the vector ALU in fp32 instead, with the same unrounded p for o, l
 *    and c.)
 *  - Results are bitwise deterministic run to run for fixed inputs.
 */
#ifndef FABFT_H
#define FABFT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  FABFT_OK = 0,
  FABFT_E_NULL = -1,     /* a required pointer is NULL */
  FABFT_E_SHAPE = -2,    /* B, H, Lq or Lk < 1, or the grid is too large, or
                            (Lk + 64) * d * 4 >= 2^32: one head's K or V
                            (Lk * d * 2 bytes) and the reads past its end
                            are addressed with 32-bit byte offsets (Lk at
                            most 8388543 at d = 128) */
  FABFT_E_HEADDIM = -3,  /* d is not 64, 96, 128 or 256 */
  FABFT_E_ALIGN = -4,    /* q, k, v or o not 16-byte aligned */
  FABFT_E_LAUNCH = -5,   /* the kernel launch failed */
  FABFT_E_SCALE = -6,    /* scale negative, NaN or infinite */
  FABFT_E_FAULT = -7,    /* fault descriptor out of range */
  FABFT_E_THRESHOLD = -8, /* threshold negative or NaN */
  FABFT_E_WORKSPACE = -9, /* workspace smaller than fabft_splitkv_workspace_bytes */
  FABFT_E_MODE = -10      /* a mode argument outside its documented values */
};

/* Detection flags, one byte per query row. */
enum {
  FABFT_FLAG_RESID = 1,     /* |pred - actual| > tau_rel * M + tau_abs, where
                               M = sum_j |O_ij| + |pred| */
  FABFT_FLAG_NONFINITE = 2, /* a residual, or the row's sum_j |O_ij| (so the
                               threshold), is NaN or infinite */
  FABFT_FLAG_WEIGHTED = 4,  /* weighted check only (fabft_set_weighted_check):
                               |pred_w - actual_w| > tau_rel * M_w + tau_abs,
                               M_w = sum_j |O_ij| + |pred_w| */
  FABFT_FLAG_SCORES = 8     /* score check only (fabft_set_score_check): see
                               there */
};

/*
 * Flash-ABFT attention forward (Algorithm 3; Eq. 8 per query row).
 * Writes O (bf16, round-to-nearest-even of the fp32 normalised output),
 * resid = pred - actual (fp32) and flags for every query row, where
 * actual = sum_j O_ij is taken from the fp32 output before bf16 rounding.
 */
int fabft_attn_fwd(const void* q, const void* k, const void* v, void* o,
                   float* resid, uint8_t* flags,
                   int B, int H, int Lq, int Lk, int d, int causal,
                   float scale);

/*
 * The same attention without the checksum (Algorithm 2): identical tiling,
 * identical O bit for bit; only the sumrow, c-update and epilogue check are
 * compiled out. Used to measure the checksum's cost.
 */
int fabft_attn_fwd_nocheck(const void* q, const void* k, const void* v,
                           void* o, int B, int H, int Lq, int Lk, int d,
                           int causal, float scale);

/*
 * The checksum hosted by Algorithm 1 instead of Algorithm 3 (Section III-B:
 * the per-query check of Eq. 8 needs only the exponentials and their sum, so
 * either algorithm can carry it). A first pass over the keys takes each
 * row's maximum score m_N (K only); a second pass accumulates o, l and
 * c = sum_k e^{s_k - m_N} sumrow_k(V) with that fixed maximum (no rescaling),
 * then O = o / l, pred = c / l and the check as in fabft_attn_fwd. Same
 * arguments, outputs, layouts, threshold and weighted check; O agrees with
 * fabft_attn_fwd to rounding (the exponentials use another reference
 * maximum), not bit for bit. Costs the Q K^T product twice. Returns
 * FABFT_E_MODE while the score check (fabft_set_score_check) is on: that
 * check runs in the one-pass kernels only.
 */
int fabft_attn_fwd_twopass(const void* q, const void* k, const void* v,
                           void* o, float* resid, uint8_t* flags,
                           int B, int H, int Lq, int Lk, int d, int causal,
                           float scale);

/*
 * The algorithm that hosts the checksum in fabft_attn_fwd, the injection and
 * debug entry points and fabft_recompute_flagged: 3 (Algorithm 3, one pass;
 * the default) or 1 (Algorithm 1, the two passes of fabft_attn_fwd_twopass),
 * so that a fault campaign can run on either form. Process-global, not
 * thread-safe. fabft_set_algorithm returns FABFT_E_MODE for any other value;
 * with Algorithm 1 selected, those entry points return FABFT_E_MODE while
 * the score check is on. The key split and fabft_attn_fwd_nocheck are not
 * affected.
 */
int fabft_set_algorithm(int alg);
int fabft_get_algorithm(void);

/*
 * Bytes of workspace that fabft_attn_fwd_splitkv needs: one partial-state
 * record of (w + 4) floats per (b, h, query row, split), w the compute width
 * (d, or 128 for d = 96). Negative status for d not 64, 96, 128 or 256, a size
 * < 1 or nsplit outside 1..64.
 */
long long fabft_splitkv_workspace_bytes(int B, int H, int Lq, int d, int nsplit);

/*
 * fabft_attn_fwd with the keys split into nsplit ranges of whole key tiles
 * (for few queries over many keys, e.g. decode): each workgroup runs
 * Algorithm 3 on one range and writes the partial state of every row
 * (running max m, l, c and the unnormalised o[d]) to the caller's workspace;
 * a merge kernel then combines the ranges with m = max_s m_s and
 * x = sum_s x_s exp(m_s - m) for x in {l, o, c} -- c merges exactly like one
 * more column of o (Eq. 10) -- and applies the per-row check after the
 * merge, so faults in the merge of o are covered too. O, resid and flags
 * have the same meaning and layout as in fabft_attn_fwd; results match it to
 * rounding (not bitwise). With Lq <= 4 the ranges run on the vector ALU
 * (every wave streams its own keys; p stays fp32 for both o and c), with
 * more rows on the matrix cores as in fabft_attn_fwd. workspace: device memory of at least
 * fabft_splitkv_workspace_bytes(B, H, Lq, d, nsplit) bytes, 16-byte aligned,
 * owned by the caller, overwritten. nsplit: 1..64. Asynchronous (two
 * launches in order on the library stream).
 */
int fabft_attn_fwd_splitkv(const void* q, const void* k, const void* v,
                           void* o, float* resid, uint8_t* flags,
                           int B, int H, int Lq, int Lk, int d, int causal,
                           float scale, int nsplit, void* workspace,
                           long long workspace_bytes);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * fabft_attn_fwd_splitkv with its per-split partial states kept in a buffer
 * that the library owns instead of a caller workspace. The buffer is a static
 * device array of FABFT_NOALLOC_SCRATCH_BYTES bytes (64 MiB), one copy per
 * GPU, held by every GPU the library runs on until the process ends; its
 * device address is looked up once per GPU, on the first call whose stream
 * belongs to that GPU. Arguments, results and validation as in
 * fabft_attn_fwd_splitkv; a problem whose workspace need
 * (fabft_splitkv_workspace_bytes) exceeds FABFT_NOALLOC_SCRATCH_BYTES returns
 * FABFT_E_WORKSPACE before anything is launched. The call allocates nothing
 * (no hipMalloc, hipFree or allocating library routine). Every call on one
 * GPU shares that GPU's buffer and leaves the last call's partial states in
 * it: calls that overlap on one GPU (other streams, other host threads)
 * race and must be serialised by the caller. Nothing in the buffer needs to
 * start at zero (every record the merge reads is written by the same call).
 * Asynchronous (two launches in order on the library stream).
 */
#define FABFT_NOALLOC_SCRATCH_BYTES (64LL << 20)
int fabft_attn_fwd_splitkv_noalloc(const void* q, const void* k, const void* v,
                                   void* o, float* resid, uint8_t* flags,
                                   int B, int H, int Lq, int Lk, int d,
                                   int causal, float scale, int nsplit);

/* Stream for all subsequent launches (a hipStream_t; NULL = null stream). */
void fabft_set_stream(void* hip_stream);

/*
 * Detection threshold: a row is flagged when NOT |r| <= tau_rel*M + tau_abs
 * (so a NaN residual is flagged). Defaults: tau_rel = 2^-16, tau_abs = 0.
 * Returns FABFT_E_THRESHOLD (and keeps the old values) for negative or NaN.
 */
int fabft_set_threshold(float tau_rel, float tau_abs);
void fabft_get_threshold(float* tau_rel, float* tau_abs);

/*
 * Score check (an extension; off by default). The output checksum cannot see
 * a fault in a score s_ik = q_i . k_k: p~, o, l and c all use the faulty
 * score consistently. With a workspace set here, every checked forward
 * (fabft_attn_fwd, the injection entry points, fabft_recompute_flagged; not
 * the key split) also compares, per query row i, the sum of its raw scores
 * over the key tiles that need no mask (all but the last one or two of a
 * causal row, and the last one when Lk % 64 != 0) with q_i . sum_k K_k over
 * the same keys (the row checksum of the product S = Q K^T), and sets
 * FABFT_FLAG_SCORES when |lhs - rhs| > tau_s * (|q_i| . sum_k |K_k|) + tau_abs.
 * The sums of K (and |K|) per key tile come from a pre-pass over K into the
 * workspace on the library stream: fabft_score_check_workspace_bytes(B, H,
 * Lk, d) bytes for a call, 16-byte aligned, caller-owned, kept in use (not
 * copied) while set; a call whose need exceeds it returns FABFT_E_WORKSPACE.
 * The masked tiles of a row (the diagonal one, a ragged last one) have no
 * such per-row prefix: there the kernel computes the tile's Q K^T a second
 * time from the same operands and sets FABFT_FLAG_SCORES when the row's
 * sums of its visible scores from the two products differ in any bit
 * (a duplicated product, not a checksum). It also catches a fault in q_i
 * that lands after the first key tile (the right-hand side uses the final
 * q_i for all full tiles); a q fault present from the start changes both
 * sides alike and is not covered.
 * d = 256 is not supported (FABFT_E_HEADDIM while the check is on).
 * workspace = NULL switches the check off. tau_s = 0 selects the default
 * (2^-22); a negative or NaN tau_s is FABFT_E_THRESHOLD. Process-global,
 * not thread-safe.
 */
long long fabft_score_check_workspace_bytes(int B, int H, int Lk, int d);
int fabft_set_score_check(void* workspace, long long workspace_bytes, float tau_s);
float fabft_get_score_threshold(void);

/*
 * Recompute on flag (after detection): for every head (b, h) with a flagged
 * row in `flags` (as written by any checked forward above on these q, k, v),
 * run the checked forward again on that head alone, up to max_retries
 * times, until none of its rows is flagged; O, resid and flags of the head
 * are overwritten by the last run. A transient fault is then corrected; a
 * head still flagged after max_retries is counted as persistent (its O is
 * not trusted). Counts go to *n_recovered and *n_persistent.
 * head_flags: device buffer of B*H bytes; head_flags_host: host buffer of
 * B*H bytes (both caller-owned scratch; the library allocates nothing).
 * Unlike the other entry points this one synchronises the library stream
 * (it needs the flags on the host). max_retries >= 1.
 */
int fabft_recompute_flagged(const void* q, const void* k, const void* v,
                            void* o, float* resid, uint8_t* flags,
                            int B, int H, int Lq, int Lk, int d, int causal,
                            float scale, uint8_t* head_flags,
                            uint8_t* head_flags_host, int max_retries,
                            int* n_recovered, int* n_persistent);

/*
 * Global check per head (Algorithm 3, the check summed over all queries of
 * the attention; the paper's single check, Eq. 5 in the per-query form of
 * Eq. 6-7): from the O and resid that fabft_attn_fwd wrote, for every
 * (b, h): gsum = sum_i resid_i = sum_i pred_i - sum_i actual_i and
 * A = sum_i sum_j |O_ij| (bf16 O), both accumulated in fp64 in a fixed order,
 * and gflags = FABFT_FLAG_RESID if NOT |gsum| <= tau_rel * A + tau_abs
 * (FABFT_FLAG_NONFINITE | FABFT_FLAG_RESID if gsum is not finite), with the
 * current threshold. o: bf16 [B, H, Lq, d] (16-byte aligned), resid: fp32
 * [B, H, Lq], gsum: fp64 [B, H], gflags: uint8 [B, H]; device pointers.
 * A fault must move its row's sum by about Lq times more than the per-row
 * check needs to be seen here. Asynchronous on the library stream.
 */
int fabft_global_check(const void* o, const float* resid, int B, int H, int Lq,
                       int d, double* gsum, uint8_t* gflags);

/*
 * Second, weighted checksum (an extension beyond the paper, which uses one
 * checksum per row): with on != 0, every checksum-on launch also carries
 *   c_w <- c_w * exp(m_old - m_new) + (sum_j (-1)^j V_kj) * p~_k
 * and compares pred_w = c_w / l with actual_w = sum_j (-1)^j O_ij, the same
 * way as the paper's check (flag FABFT_FLAG_WEIGHTED). A fault on p~_k after
 * the checksum read it moves actual by delta * sumrow_k(V) / l, which the
 * paper's check misses when sumrow_k(V) is near 0; the weighted sum of that
 * V row is then usually far from 0. Default: off. Process-global, not
 * thread-safe. resid stays the paper's residual pred - actual.
 */
void fabft_set_weighted_check(int on);
int fabft_get_weighted_check(void);

/*
 * Persistent workgroups (a launch shape, not part of the method). When on,
 * fabft_attn_fwd and fabft_attn_fwd_nocheck launch only as many workgroups
 * as the device holds at once (one per compute unit) when
 * there are more (head, query tile) items than that, each workgroup running
 * a fixed list of items; the next item's Q and first key tiles load while
 * the current item's last tiles and its epilogue run. It applies without the
 * mask, or with it when B * H is a multiple of 8, and never to the split,
 * debug, injection or score-check paths. Results are bitwise the same
 * either way (each row is computed by the same instructions in the same
 * order). Modes: FABFT_PERSIST_OFF (one workgroup per item),
 * FABFT_PERSIST_AUTO (default: on for d = 64, 96 and 128 when Lk <= 1024,
 * where a workgroup's start-up is a large part of its work),
 * FABFT_PERSIST_ALWAYS.
 * fabft_set_persistent returns FABFT_E_MODE for any other value.
 * Process-global, not thread-safe.
 */
enum { FABFT_PERSIST_OFF = 0, FABFT_PERSIST_AUTO = 1, FABFT_PERSIST_ALWAYS = 2 };
int fabft_set_persistent(int mode);
int fabft_get_persistent(void);

/* Number of keys per key tile of the kernel for head dimension d (the unit
 * of fabft_fault.tile at the O site), or FABFT_E_HEADDIM. */
int fabft_key_tile(int d);

/* Number of query rows per workgroup for head dimension d (the unit of
 * fabft_fault.tile at the V and VS sites): 256 at d = 64, 96 and 128, 128
 * at d = 256; FABFT_E_HEADDIM for an unsupported d. */
int fabft_query_tile(int d);

/* Fault sites for the injection path (where a single bit is flipped). */
enum {
  FABFT_SITE_NONE = 0, /* no fault: debug run returning pred and actual */
  FABFT_SITE_S = 1,    /* fp32 score s_ik after Q K^T, before the row max */
  FABFT_SITE_P = 2,    /* bf16 weight p~_ik after the checksum has read it,
                          before the P V product */
  FABFT_SITE_O = 3,    /* fp32 output accumulator o_ij right after the
                          P V product of key tile `tile` */
  FABFT_SITE_V = 4,    /* bf16 V_kj in the on-chip copy of one workgroup,
                          after sumrow_k(V) was taken, before the P V product
                          reads it; every query row of that workgroup that
                          sees key k reads the flipped value */
  /* checker state (Section IV-B counts faults there as possible false
     positives): */
  FABFT_SITE_C = 5,    /* fp32 checksum accumulator pair c = c_hi + c_lo of
                          query row `row` (col 0: c_hi, col 1: c_lo) after
                          the update of key tile `tile`. c and l of a row
                          are held as two partial sums, one per half of the
                          keys (keys k with k mod 16 < 8, and the others),
                          added at the end; this site flips the first half's
                          register */
  FABFT_SITE_L = 6,    /* fp32 accumulator l of the row after key tile
                          `tile` (the first key half's partial sum, as for
                          FABFT_SITE_C) */
  FABFT_SITE_M = 7,    /* fp32 running max (scale * log2 e units) of the row,
                          as held by the lane of the row's first key half,
                          after the exponentials of key tile `tile` */
  FABFT_SITE_Q = 8,    /* bf16 q_ij in the registers of query row `row`
                          (col = j), flipped before the Q K^T of key tile
                          `tile`; the flipped value stays for the later tiles
                          (a register fault; upstream of o, l and c alike) */
  FABFT_SITE_VS = 9    /* checker state: the bf16 sumrow(V) operand of key
                          `row` (col 0: high part, col 1: low part) in the
                          copy of one workgroup (tile = query tile, as for V) */
};

/* Most faults one injection launch takes (fabft_attn_fwd_inject_n). */
#define FABFT_MAX_FAULTS 8

/*
 * One single-bit fault. b, h select the head. For S and P: row = query i,
 * col = key k (must be visible to i). For O: row = query i, col = output
 * column j, tile = key tile index t (the fault lands after tile t; t must be
 * a tile that row i processes: t*key_tile <= last visible key of i). For V:
 * row = key k, col = column j, tile = query tile (rows tile*query_tile ..
 * tile*query_tile + query_tile - 1) whose workgroup holds the flipped copy.
 * For C: row = query i, col 0 or 1, tile as for O. For L, M: row = query i,
 * col = 0, tile as for O. For Q: row = query i,
 * col = j < d, tile as for O. For VS: row = key k, col 0 or 1, tile as for V.
 * bit: 0..31 for fp32 sites (S, O, C, L, M), 0..15 for bf16 sites (P, V, Q,
 * VS).
 */
typedef struct {
  int site, b, h, row, col, tile, bit;
} fabft_fault;

/*
 * Debug / fault-injection variant of fabft_attn_fwd (a separate kernel
 * instantiation; the production kernels carry no injection code).
 * f may be NULL (same as site NONE). pred, actual, pred_w and actual_w may
 * be NULL; when given, they receive c/l and sum_j O_ij per row, and with the
 * weighted check on, c_w/l and sum_j (-1)^j O_ij (0 when it is off); all
 * fp32 [B, H, Lq]. Returns FABFT_E_FAULT if the descriptor is out of range.
 * Asynchronous.
 */
int fabft_attn_fwd_inject(const void* q, const void* k, const void* v,
                          void* o, float* resid, uint8_t* flags,
                          int B, int H, int Lq, int Lk, int d, int causal,
                          float scale, const fabft_fault* f,
                          float* pred, float* actual,
                          float* pred_w, float* actual_w);

/*
 * The same with a list of faults applied in one launch (the paper's runs
 * with several faults): faults[0 .. nfaults-1], each checked as above;
 * entries with site FABFT_SITE_NONE are skipped. 0 <= nfaults <=
 * FABFT_MAX_FAULTS (else FABFT_E_FAULT); faults may be NULL when nfaults is
 * 0. Faults at the same element and time flip that bit once per entry, in
 * list order.
 */
int fabft_attn_fwd_inject_n(const void* q, const void* k, const void* v,
                            void* o, float* resid, uint8_t* flags,
                            int B, int H, int Lq, int Lk, int d, int causal,
                            float scale, const fabft_fault* faults, int nfaults,
                            float* pred, float* actual,
                            float* pred_w, float* actual_w);

/*
 * Optional per-row debug outputs of fabft_attn_fwd_debug; each pointer may be
 * NULL (not written), else fp32 [B, H, Lq] on the device.
 *  pred, actual      c / l (Eq. 8) and sum_j O_ij (fp32, before rounding)
 *  pred_w, actual_w  the weighted check's c_w / l and sum_j (-1)^j O_ij
 *                    (0 while the weighted check is off)
 *  score_lhs         the score check's sum of the row's raw scores q_i . k_k
 *                    over the key tiles without a mask (see
 *                    fabft_set_score_check), as they entered the softmax
 *  score_rhs         q_i . sum_k K_k over the same keys (the q_i held at the
 *                    end of the pass)
 *  score_bound       |q_i| . sum_k |K_k| over the same keys (the threshold is
 *                    tau_s times it)
 * The three score outputs are 0 while the score check is off. Section II's
 * row checksum of a matrix product, applied to S = Q K^T.
 */
typedef struct {
  float* pred;
  float* actual;
  float* pred_w;
  float* actual_w;
  float* score_lhs;
  float* score_rhs;
  float* score_bound;
} fabft_debug_out;

/*
 * Debug / fault-injection forward with every debug output: the same
 * computation and fault list as fabft_attn_fwd_inject_n (the injection
 * instantiation), writing the outputs `out` selects (out may be NULL).
 * Asynchronous.
 */
int fabft_attn_fwd_debug(const void* q, const void* k, const void* v,
                         void* o, float* resid, uint8_t* flags,
                         int B, int H, int Lq, int Lk, int d, int causal,
                         float scale, const fabft_fault* faults, int nfaults,
                         const fabft_debug_out* out);

/* Human-readable text for a status code (static storage). */
const char* fabft_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* FABFT_H */
