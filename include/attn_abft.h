/*
 * attn_abft.h - C ABI of the ABFT-protected multi-head attention layer
 * (EEC-ABFT, ATTNChecker: arXiv 2410.11720) on AMD MI355X (gfx950).
 *
 * The layer (paper Sec. 2.1, Eq. 1-2, Fig. 1) with GPT-2 style packed
 * weights:
 *   [Q | K | V] = X Wqkv,  AS_h = Q_h K_h^T,  AP_h = softmax(scale * AS_h [causal mask]),
 *   CL_h = AP_h V_h,       O = CL Wo,
 * and its backward. Every GEMM output carries unweighted and weighted
 * checksums (weights 1..R inside R-row blocks, Sec. 2.3) that are encoded
 * once per protection section and passed through the section's GEMMs
 * (Sec. 4.4), then verified with EEC-ABFT (Sec. 4.2, 4.3): INF, NaN and
 * near-INF errors are detected, located and corrected in place.
 *
 * Conventions for every entry point
 * ---------------------------------
 * - Pointers marked (device) are caller-owned device memory on the current
 *   HIP device; the library allocates nothing, creates no stream or event,
 *   and keeps no state between calls beyond read-only facts about each
 *   device it has run on (its architecture and the number of compute
 *   units per XCD, read once). Pointers marked (host) are read during the
 *   call only.
 * - `stream` is a hipStream_t (NULL = the null stream). All GPU work of a
 *   call is enqueued asynchronously on it and on no other stream; outputs
 *   and the report are valid after the caller synchronises the stream.
 * - Layouts are dense row-major (C order), dimensions listed outermost first.
 * - bf16 storage is IEEE bfloat16 (round-to-nearest-even when produced);
 *   accumulation and all checksums are fp32.
 * - Return value: ABFT_OK, or a negative status covering argument and
 *   launch errors only. On an argument error nothing is enqueued. Detected,
 *   corrected and uncorrectable faults are NOT status codes: they are
 *   reported in the abft_report (device) and read after a sync;
 *   n_uncorrectable > 0 is the caller's cue to fall back to
 *   checkpoint/restore.
 */
#ifndef ATTN_ABFT_H
#define ATTN_ABFT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------- */
#define ABFT_OK               0
#define ABFT_ERR_INVALID     -1   /* null pointer, bad shape, R does not divide seq, ... */
#define ABFT_ERR_UNSUPPORTED -2   /* dtype / mode not implemented, not a gfx950 device */
#define ABFT_ERR_HIP         -3   /* a kernel launch failed */
#define ABFT_ERR_WORKSPACE   -4   /* workspace smaller than attn_abft_workspace_bytes() */

/* ---- storage dtypes -------------------------------------------------- */
#define ABFT_BF16 0
#define ABFT_FP32 1

/* ---- protection sections (Sec. 4.4), the per-step enable mask that the
 *      adaptive frequencies of Sec. 4.5 act on ---------------------------- */
#define ABFT_SEC_AS  1u   /* X W^Q, X W^K, Q K^T            */
#define ABFT_SEC_CL  2u   /* X W^V, AP V                    */
#define ABFT_SEC_O   4u   /* CL W^O                         */
#define ABFT_SEC_BWD 8u   /* every backward GEMM            */
#define ABFT_SEC_ALL 15u

/* ---- flags ----------------------------------------------------------- */
#define ABFT_FLAG_ROOT_CHECK    1u  /* verify Q, K, V right after the projection */
#define ABFT_FLAG_REPORT_APPEND 2u  /* keep the report's contents at entry        */
#define ABFT_FLAG_UNPROTECTED   4u  /* no checksums and no verification: the same
                                       kernels without ABFT (overhead baseline)  */
#define ABFT_FLAG_FUSED         8u  /* forward: score, softmax and context in one
                                       kernel that stores neither AS nor AP (an
                                       extension of Sec. 4.4: AS checked on its
                                       row side per R-key block against
                                       Q (K^c)^T, CL against the V^r row
                                       checksum carried through the online
                                       softmax; CL^c summed in the kernel
                                       from the checked, stored CL; Q verified at the projection even
                                       without ABFT_FLAG_ROOT_CHECK, fixed from
                                       its checksums then, as the row side
                                       cannot see a Q error). Needs bf16
                                       storage and seq a multiple of 128 (else
                                       ABFT_ERR_UNSUPPORTED); the stage bits
                                       SCORE, SOFTMAX and CONTEXT each select
                                       that kernel. It saves each query's
                                       softmax max and sum and CL^r. A backward
                                       with the same flag runs a fused core in
                                       place of dAP, the softmax backward and
                                       the dQ, dK and dV GEMMs, storing no
                                       score-shaped tensor (the workspace holds
                                       none: attn_abft_workspace_bytes is
                                       smaller): a query pass (stage bits
                                       SOFTMAX_BWD, DQ) recomputes
                                       S = Q K^T, row-checked per (query, R-key
                                       block) against Q (K^c)^T, takes P from
                                       the statistics, dP = dCL V^T row-checked
                                       against dCL (V^c)^T, dS = scale P (dP -
                                       D) with D = dCL . CL, and dQ = dS K
                                       row-checked against dS K^r; a key pass
                                       (bits DV, DK) recomputes S and dP again,
                                       column-checked per (R-query block, key)
                                       against (Q^c) K^T and (dCL^c) V^T, and
                                       forms dV = P^T dCL and dK = dS^T Q,
                                       row-checked against P^T dCL^r and
                                       dS^T Q^r (CORE_BWD selects both; each
                                       pass forms the row checksums K^r, Q^r
                                       and dCL^r over each head's dims from
                                       the tiles it loads).
                                       A located dQ, dK or dV element is fixed
                                       from the checksum. AS faults reach both
                                       passes' recomputed scores (two events),
                                       dAP faults both passes' dP. */

/* ---- op tags of protected GEMM outputs (paper Table 1 + backward) ----- */
enum abft_op {
  ABFT_OP_Q = 0, ABFT_OP_K, ABFT_OP_V, ABFT_OP_AS, ABFT_OP_CL, ABFT_OP_O,
  ABFT_OP_DCL, ABFT_OP_DWO, ABFT_OP_DAP, ABFT_OP_DV, ABFT_OP_DQ, ABFT_OP_DK,
  ABFT_OP_DWQ, ABFT_OP_DWK, ABFT_OP_DWV, ABFT_OP_DX, ABFT_NUM_OPS
};
/* extreme-value class of a located element (Sec. 2.2) */
enum abft_kind { ABFT_KIND_NUMERIC = 0, ABFT_KIND_NEAR_INF = 1, ABFT_KIND_INF = 2,
                 ABFT_KIND_NAN = 3, ABFT_KIND_NONE = 4 };
/* what was done about it */
enum abft_action { ABFT_ACT_RECOMPUTE = 0, ABFT_ACT_DELTA = 1, ABFT_ACT_RECONSTRUCT = 2,
                   ABFT_ACT_UNCORRECTABLE = 3 };

/* Coordinates (b, h, row, col) of an element of op's output:
 *   Q K V CL dCL dV dQ dK : b, head h, token row in [0,seq), col in [0,head_dim)
 *   AS dAP                : b, head h, query row, key col (both in [0,seq))
 *   O dX                  : b, h = 0, token row, col in [0,hidden)
 *   dWO dWQ dWK dWV       : b = h = 0, row in [0,hidden) (input feature),
 *                           col in [0,hidden) (output feature of that block)
 * For an UNCORRECTABLE event of a column vector, row is the first row of
 * its checksum block; of a row vector, col is the first column of its block. */

typedef struct {
  int32_t batch, seq, hidden, heads; /* hidden = heads * head_dim            */
  int32_t dtype;                     /* ABFT_BF16 | ABFT_FP32 (activation storage) */
  int32_t causal;                    /* 1: key j > query i is masked          */
  int32_t block_rows;                /* R: checksum block on token axes; a power
                                        of two, 16 <= R <= 128, R | seq        */
  float   scale;                     /* softmax scale; <= 0 -> 1/sqrt(head_dim) */
  float   t_near_inf;                /* Sec. 4.2, default 1e10 (compared as stored) */
  float   t_correct;                 /* Sec. 4.2, default 1e5                   */
  float   e_rel;                     /* detection bound E = e_rel * sum|v|; 0 ->
                                        2^-4 (bf16) / 2^-13 (fp32)              */
  uint32_t sections;                 /* ABFT_SEC_* enabled this call; a forward
                                        whose backward is protected must have
                                        ABFT_SEC_BWD set (it saves the checksums
                                        the backward propagates)                */
  uint32_t flags;                    /* ABFT_FLAG_*                             */
} attn_abft_config;

/* One injected fault (test-only injector, Sec. 5.1), applied to element
 * (b, h, row, col) of op's output after the output is rounded to storage
 * and before it is verified:
 *   mode ABFT_FAULT_SET:  overwritten with `value` rounded to storage;
 *   mode ABFT_FAULT_FLIP: the most significant exponent bit of the stored
 *                         value is flipped (bit 14 of bf16, bit 30 of fp32;
 *                         `value` is ignored) - the paper's way of making a
 *                         near-INF value from a computed one. */
#define ABFT_FAULT_SET  0
#define ABFT_FAULT_FLIP 1
typedef struct { int32_t op, b, h, row, col; float value; int32_t mode; } abft_fault;

typedef struct {
  int32_t op, b, h, row, col, kind, action, reserved;
  float observed;                    /* the stored value that was located    */
  float reserved2;
} abft_event;

typedef struct {
  int32_t n_events;                  /* events appended (may exceed capacity) */
  int32_t n_corrected;
  int32_t n_uncorrectable;
  int32_t capacity;                  /* set by attn_abft_report_init          */
  int32_t overflow;                  /* 1 if events were dropped              */
  int32_t reserved[3];
  abft_event events[];               /* capacity entries, unordered          */
} abft_report;

/* Bytes of device workspace attn_abft_forward needs and attn_abft_backward
 * reuses (saved Q/K/V, AP, CL, propagated checksums and backward scratch).
 * 0 if the config is invalid. */
size_t attn_abft_workspace_bytes(const attn_abft_config* cfg /* host */);

/* Bytes of a report able to hold `capacity` events. */
size_t attn_abft_report_bytes(int32_t capacity);

/* Initialise a report (device) for `capacity` events: zero counters, set
 * capacity. Must be called once after allocating it. */
int attn_abft_report_init(abft_report* report, int32_t capacity, void* stream);

/* Protected forward (Sec. 4.4).
 *   X    [batch, seq, hidden]    (device, dtype)
 *   Wqkv [hidden, 3*hidden]      (device, dtype)  Q|K|V column blocks
 *   Wo   [hidden, hidden]        (device, dtype)
 *   O    [batch, seq, hidden]    (device, dtype)  output
 *   workspace (device, >= attn_abft_workspace_bytes) receives the saved
 *   tensors; it must stay untouched until the matching backward.
 *   faults (device) n_faults entries, may be NULL when n_faults == 0.
 *   report (device) initialised report; reset at entry unless
 *   ABFT_FLAG_REPORT_APPEND. */
int attn_abft_forward(const attn_abft_config* cfg, const void* X, const void* Wqkv,
                      const void* Wo, void* O, void* workspace, size_t workspace_bytes,
                      const abft_fault* faults, int32_t n_faults, abft_report* report,
                      void* stream);

/* Protected backward (extension: every backward GEMM output gets a
 * propagated column checksum and a column pass).
 *   dO [batch, seq, hidden] (device, dtype); X, Wqkv, Wo as in forward;
 *   workspace: the one the forward filled (its backward scratch is reused);
 *   dX [batch, seq, hidden] (device, dtype); dWqkv [hidden, 3*hidden] and
 *   dWo [hidden, hidden] (device, fp32). */
int attn_abft_backward(const attn_abft_config* cfg, const void* dO, const void* X,
                       const void* Wqkv, const void* Wo, void* workspace,
                       size_t workspace_bytes, void* dX, float* dWqkv, float* dWo,
                       const abft_fault* faults, int32_t n_faults, abft_report* report,
                       void* stream);

/* Allocation-free protected forward, for callers that cannot allocate
 * device memory (code under graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): attn_abft_forward with ABFT_FLAG_FUSED (required,
 * else ABFT_ERR_UNSUPPORTED), its workspace replaced by a buffer of 64 MiB
 * that the library holds on every device it runs on until the process
 * ends; no memory is allocated during the call. Arguments as for
 * attn_abft_forward; nothing is saved for a backward (ABFT_SEC_BWD is
 * ignored). The layer must fit the buffer: T = batch * seq tokens need
 * about T * hidden * 8 bytes (storage bf16) plus T * heads * 32 bytes and
 * (T / block_rows) * hidden * 56 bytes of checksums, their bf16 images and
 * softmax statistics (B8 S1024 H768 with 12 heads: 56 MB);
 * a larger layer returns ABFT_ERR_WORKSPACE before anything is enqueued.
 * Every call on a device shares that device's buffer and leaves its
 * contents behind: calls that overlap on one device (other streams, other
 * host threads) race and must be serialised by the caller. */
int attn_abft_forward_noalloc(const attn_abft_config* cfg, const void* X, const void* Wqkv,
                              const void* Wo, void* O, const abft_fault* faults,
                              int32_t n_faults, abft_report* report, void* stream);

/* Stages of the chains, for profiling one kernel at a time with
 * attn_abft_forward_stages / attn_abft_backward_stages. */
#define ABFT_STAGE_ENCODE      0x001u  /* checksum encoders (fwd: W^V, X; bwd: dO) */
#define ABFT_STAGE_QKV         0x002u  /* fwd: [Q|K|V] = X Wqkv                     */
#define ABFT_STAGE_SCORE       0x004u  /* fwd: AS = Q K^T                           */
#define ABFT_STAGE_SOFTMAX     0x008u  /* fwd: AP = softmax(scale AS)               */
#define ABFT_STAGE_CONTEXT     0x010u  /* fwd: CL = AP V                            */
#define ABFT_STAGE_OUT         0x020u  /* fwd: O = CL Wo (fused: CL^c from the fused kernel) */
#define ABFT_STAGE_DCL         0x002u  /* bwd: dCL = dO Wo^T                        */
#define ABFT_STAGE_DWO         0x004u  /* bwd: dWo = CL^T dO                        */
#define ABFT_STAGE_DAP         0x008u  /* bwd: dAP = dCL V^T (fused: no work)       */
#define ABFT_STAGE_DV          0x010u  /* bwd: dV = AP^T dCL (fused: the key pass)  */
#define ABFT_STAGE_SOFTMAX_BWD 0x020u  /* bwd: dAS = scale AP (dAP - rowdot)
                                          (fused: the query pass)               */
#define ABFT_STAGE_DQ          0x040u  /* bwd: dQ = dAS K (fused: the query pass)   */
#define ABFT_STAGE_DK          0x080u  /* bwd: dK = dAS^T Q (fused: the key pass)   */
#define ABFT_STAGE_DWQKV       0x100u  /* bwd: dWqkv = X^T [dQ|dK|dV]               */
#define ABFT_STAGE_DX          0x200u  /* bwd: dX = [dQ|dK|dV] Wqkv^T (fused:
                                          [dQ|dK|dV]^c encoded first)           */
#define ABFT_STAGE_CORE_BWD    0x400u  /* bwd after a fused forward: the whole
                                          fused backward core                   */
#define ABFT_STAGE_ALL         0x7ffu

/* attn_abft_forward / attn_abft_backward restricted to the stages in the
 * mask (profiling). A stage reads what earlier stages left in the
 * workspace, so a full call on the same workspace must come first; the
 * report is reset at entry unless ABFT_FLAG_REPORT_APPEND. Arguments and
 * errors as for the full calls. */
int attn_abft_forward_stages(const attn_abft_config* cfg, const void* X, const void* Wqkv,
                             const void* Wo, void* O, void* workspace, size_t workspace_bytes,
                             const abft_fault* faults, int32_t n_faults, abft_report* report,
                             uint32_t stages, void* stream);
int attn_abft_backward_stages(const attn_abft_config* cfg, const void* dO, const void* X,
                              const void* Wqkv, const void* Wo, void* workspace,
                              size_t workspace_bytes, void* dX, float* dWqkv, float* dWo,
                              const abft_fault* faults, int32_t n_faults, abft_report* report,
                              uint32_t stages, void* stream);

/* Checksum encoder (Sec. 4.6, "Encoding"). A is `batch` matrices of
 * rows x cols (element (b, i, j) at A + b*batch_stride + i*ld + j, in
 * elements of dtype). Writes, when the pointer is not NULL,
 *   col_chk [batch][rows/block_rows][2][cols]  unweighted and weighted
 *           (weights 1..block_rows) sums of every column in each row block,
 *   row_chk [batch][rows][cols/block_cols][2]  the same along rows,
 * both fp32 (device). block_rows | rows, block_cols | cols. */
int encode_checksums(const void* A, int32_t dtype, int64_t batch, int64_t rows, int64_t cols,
                     int64_t ld, int64_t batch_stride, int32_t block_rows, int32_t block_cols,
                     float* col_chk, float* row_chk, void* stream);

/* Standalone EEC-ABFT detection and correction (Sec. 4.2, 4.3) of C
 * (device, same addressing as encode_checksums) against propagated
 * checksums in the encode_checksums layouts. col_chk is required; with
 * row_chk also given the column pass is followed by the row pass and the
 * checksum refresh of Sec. 4.3. With no operands at hand, located elements
 * are corrected from the checksums (DELTA if |d1| <= t_correct, else
 * RECONSTRUCT); events carry op_tag, b = batch index, h = 0. t_near_inf is
 * compared as stored in dtype; e_rel as in attn_abft_config (0 = default).
 * The report is appended to. */
int verify_and_correct(void* C, int32_t dtype, int64_t batch, int64_t rows, int64_t cols,
                       int64_t ld, int64_t batch_stride, int32_t block_rows, int32_t block_cols,
                       float* col_chk, float* row_chk, float t_near_inf, float t_correct,
                       float e_rel, int32_t op_tag, abft_report* report, void* stream);

/* Byte offsets of the saved tensors inside the workspace (for inspection):
 * QKV [batch, seq, 3*hidden] dtype, AP [batch, heads, seq, seq] dtype
 * (only blocks with key block <= query block are written under a causal
 * mask), CL [batch, seq, hidden] dtype. Returns ABFT_OK, ABFT_ERR_INVALID,
 * or ABFT_ERR_UNSUPPORTED when ap_offset is requested for a config with
 * ABFT_FLAG_FUSED (that workspace holds no AP). */
int attn_abft_workspace_offsets(const attn_abft_config* cfg, size_t* qkv_offset,
                                size_t* ap_offset, size_t* cl_offset);

/* Human-readable text of a status code (static storage). */
const char* attn_abft_strerror(int status);

/* Byte offset inside the workspace of a tensor the forward or backward
 * leaves there (for inspection; row-major):
 *   which = 0: QKV [B, S, 3H]; 1: AS [B, nh, S, S] (valid from the forward
 *   until the next backward, which reuses its space for dAP); 2: AP
 *   [B, nh, S, S]; 3: CL [B, S, H]; 4: dQKV [B, S, 3H] (backward: dQ|dK|dV);
 *   5: dCL [B, S, H] (backward); 8: dAS [B, nh, S, S] (backward): storage
 *   dtype. 6: AP^c [B, nh, S/R, 2, S] and 7: AP^r [B, nh, S, S/R, 2]: fp32
 *   column and row checksums of the stored AP (unweighted, weighted) per
 *   R-query and R-key block.
 * Under a causal mask the score-shaped tensors hold meaningful values only
 * on the pairs the mask allows (key <= query); other positions are zero
 * where written and unspecified elsewhere. With ABFT_FLAG_FUSED the
 * score-shaped tensors (1, 2, 6, 7, 8) do not exist: ABFT_ERR_UNSUPPORTED.
 * Returns ABFT_ERR_INVALID for an invalid config or `which`. */
int attn_abft_workspace_tensor(const attn_abft_config* cfg, int32_t which, size_t* offset);

/* ---------------------------------------------------------------------------
 * Adaptive detection frequencies (paper Sec. 4.5, Algorithm 1). Host-only
 * calls (no device memory, no stream): they choose how often each
 * protection section is checked and produce the `sections` mask of a
 * training step.
 *
 * Coverage model: errors of type e (INF, NaN, near-INF, in this order)
 * strike an operation of n flops as a Poisson process of rate lambda[e]
 * per flop; a section survives no error, or exactly one error that is
 * either handled (its checks run, a fraction f of the steps) or harmless
 * (probability 1 - p[e], p from the paper's Table 4: the chance that one
 * error of that type in that operation leads to a non-trainable state).
 * Two or more errors in one section count as failure. The failure
 * probability of one execution is U = 1 - prod_S FC_S(f_S).
 * ------------------------------------------------------------------------- */
typedef struct {
  double flops;   /* n: flops of the operation per execution (>= 0)          */
  double p[3];    /* P(non-trainable | one error of type INF, NaN, near-INF) */
} abft_freq_op;

typedef struct {
  int32_t n_ops;     /* operations in the section                            */
  int32_t first_op;  /* index of its first operation in the op array         */
  double  cost;      /* T_S: check time of the section when run every step   */
} abft_freq_section;

/* Failure probability per execution for frequencies freqs[n_secs] (each in
 * [0, 1]). ops/secs/lambda[3]/freqs (host). n_secs in [1, 16]. Returns
 * ABFT_ERR_INVALID for null pointers or values out of range. */
int attn_abft_unsafe_probability(const abft_freq_op* ops, const abft_freq_section* secs,
                                 int32_t n_secs, const double* lambda, const double* freqs,
                                 double* unsafe_out);

/* Algorithm 1: frequencies f_S (freqs_out[n_secs], host) that minimise the
 * check time sum f_S T_S subject to a failure probability of at most
 * fail_target (= 1 - FC_target) per execution. Sections are filled in
 * descending order of coverage gained per unit of check time, wholly while
 * the remaining deficit allows and then by the fraction that closes it
 * (the greedy optimum of the first-order expansion of the product). A
 * target that even full checking misses returns all ones. */
int attn_abft_optimize_frequencies(const abft_freq_op* ops, const abft_freq_section* secs,
                                   int32_t n_secs, const double* lambda, double fail_target,
                                   double* freqs_out);

/* The attn_abft_config.sections mask for training step `step` (>= 0) given
 * the frequencies of S_AS, S_CL, S_O and S_BWD (freqs[4], host): section S
 * is on when floor((step + 1) f_S) > floor(step f_S), i.e. on a fraction
 * f_S of the steps, evenly spread (f >= 1: every step; f <= 0: never). The
 * same mask must be used for the forward and the backward of the step. */
uint32_t attn_abft_sections_for_step(const double* freqs, int64_t step);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_ABFT_H */
