// Internal declarations shared by the kernels and the host orchestration of
// the ABFT-protected attention layer. Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_abft.h"

namespace abft {

enum class Layout : int { KMajor = 0, MNMajor = 1 };

// How a protected GEMM maps its output element (z, m, n) to the event
// coordinates (op, b, h, row, col) of the public ABI:
//   op  = op_base + n / op_span,   nn = n % op_span
//   z-batched (nb1 > 0): b = z / nb1, h = z % nb1, row = m, col = nn
//   token-major       : b = m / rows_per_b, row = m % rows_per_b (or b = 0,
//                       row = m when rows_per_b == 0); h = nn / head_cols,
//                       col = nn % head_cols (or h = 0, col = nn).
struct CoordMap {
  int op_base = 0;
  int op_span = 1 << 30;
  int nb1 = 0;
  int rows_per_b = 0;
  int head_cols = 0;
};

// C[z](m, n) = sum_k A[z](m, k) * B[z](k, n) with z = b0 * nb1 + b1.
// Element addresses (in elements of the storage type):
//   A(m,k): A + b0*sA0 + b1*sA1 + (A K-major ? m*lda + k : k*lda + m)
//   B(k,n): B + b0*sB0 + b1*sB1 + (B K-major ? n*ldb + k : k*ldb + n)
//   C(m,n): C + b0*sC0 + b1*sC1 + m*ldc + n
// Column-checksum side (paper Sec. 2.3 A^c, carried as extra MFMA rows):
//   Ac(r,k) fp32, r in [0, 2M/Rm): laid out like A (K-major: r*ldac + k)
//   Cc(r,n) fp32 optional store of the propagated C^c = A^c B
// (Rm and Rn, the checksum block sizes, are powers of two.)
// Row-checksum side (B^r, extra MFMA columns), for columns n >= cr_n_begin:
//   Br(k,q) fp32, q in [0, 2(N - cr_n_begin)/Rn): laid out like B
//   Cr(m,q) fp32 optional store of the propagated C^r = A B^r
struct GemmDesc {
  int M = 0, N = 0, K = 0;
  int nb0 = 1, nb1 = 1;
  const void* A = nullptr; int64_t lda = 0, sA0 = 0, sA1 = 0;
  const void* B = nullptr; int64_t ldb = 0, sB0 = 0, sB1 = 0;
  void* C = nullptr; int64_t ldc = 0, sC0 = 0, sC1 = 0;

  const float* Ac = nullptr; int64_t ldac = 0, sAc0 = 0, sAc1 = 0;
  // optional bf16 image of Ac for an unbatched A (either layout): per
  // checksum block four rows (c1 hi, c1 lo, c2 hi, c2 lo, hi = bf16(c), lo
  // = bf16(c - hi)) along k, each ldaci elements long; the direct-to-LDS
  // path then copies the column strip like an operand tile
  const uint16_t* Aci = nullptr; int64_t ldaci = 0;
  float* Cc = nullptr; int64_t ldcc = 0, sCc0 = 0, sCc1 = 0;
  int Rm = 128;

  const float* Br = nullptr; int64_t ldbr = 0, sBr0 = 0, sBr1 = 0;
  // optional bf16 image of Br for an unbatched B, laid out like Aci (four
  // rows per checksum block along k, ldbri elements each)
  const uint16_t* Bri = nullptr; int64_t ldbri = 0;
  float* Cr = nullptr; int64_t ldcr = 0, sCr0 = 0, sCr1 = 0;
  int Rn = 128;
  int cr_n_begin = 0;

  // 0: dense; 1: skip tiles strictly above the block diagonal (score-shaped
  // outputs, key > query); 2: K range ends at the tile's last row (A is a
  // masked probability matrix, keys <= query); 3: K range starts at the
  // tile's first row (A is the transpose of such a matrix).
  int causal = 0;
  // 0: no verification; 1: column pass; 2: column pass, row pass and the
  // checksum refresh of Sec. 4.3 (two-sided outputs).
  int verify = 0;
  int verify_n_lo = 0, verify_n_hi = 1 << 30;  // only columns in [lo, hi) are verified
  int recompute = 1;  // correct by recomputing from A and B, else from checksums
  float e_rel = 0.f, tn = 0.f, tc = 0.f;
  CoordMap map;
  const abft_fault* faults = nullptr;
  int n_faults = 0;
  abft_report* report = nullptr;
  // Split-K (dense, unbatched, fp32 output only): the workgroup of K slice
  // kz writes raw fp32 partials to C + kz*sCk and C^c to Cc + kz*sCck,
  // without rounding, faults or verification; launch_splitk_reduce sums the
  // slices and verifies.
  int splitk = 1;
  int64_t sCk = 0, sCck = 0;
};

// Tile shapes the GEMM is instantiated for (S1: one LDS stage, for short K
// such as the head dimension, so that more workgroups fit on a CU).
enum class Tile : int { T128x128 = 1, T128x64 = 2, T128x128S1 = 3 };

// Launch one protected (or, with no checksum operands, plain) GEMM.
// dtype: ABFT_BF16 or ABFT_FP32 operands; c_fp32: output stored as fp32.
hipError_t launch_gemm(const GemmDesc& g, int dtype, bool c_fp32, Layout la, Layout lb,
                       Tile tile, hipStream_t stream);

// A weight gradient w (MN-major operands, fp32 output, whole or as its K
// slices, as launch_gemm takes it) and a projection p (K-major operands,
// bf16 output, 128 x 128 tiles) in one launch, when both take the direct
// path and w's workgroups are a multiple of 8; hipErrorNotSupported when
// they do not qualify (nothing launched: launch them one by one).
hipError_t launch_gemm_pair(const GemmDesc& w, const GemmDesc& p, int dtype,
                            hipStream_t stream);

// Sum the split-K partials of a protected GEMM (fixed order), apply
// injected faults, run the column pass (recompute correction from A and B)
// and store C. g describes the full GEMM with its final C, Rm, map, faults
// and report; P and Pc are the partials the split launch wrote.
hipError_t launch_splitk_reduce(const GemmDesc& g, const float* P, const float* Pc, int dtype,
                                Layout la, Layout lb, hipStream_t stream);

// Softmax over keys with checksum carry-through (fwd) and its backward.
struct SoftmaxDesc {
  int B = 0, nh = 0, S = 0, R = 128;
  int causal = 0;
  // Under a causal mask a query block's row is produced up to the end of
  // the score-GEMM tile holding its diagonal (keys past the diagonal are
  // written as exact zeros), so the consumers' K ranges only read written
  // data.
  int kv_align = 128;
  float scale = 1.f;
  const void* AS = nullptr;   // [B,nh,S,S] fwd input (unscaled scores)
  void* AP = nullptr;         // [B,nh,S,S] fwd output / bwd input
  const void* dAP = nullptr;  // [B,nh,S,S] bwd input
  void* dAS = nullptr;        // [B,nh,S,S] bwd output
  float* col_chk = nullptr;   // [B,nh,S/R,2,S] of the produced matrix (may be null)
  float* row_chk = nullptr;   // [B,nh,S,S/R,2] of the produced matrix (may be null)
  // CUs per XCD of the device (set by the launcher; 0 keeps the plain
  // workgroup order)
  int xcd_cus = 0;
};
hipError_t launch_softmax_fwd(const SoftmaxDesc& d, int dtype, hipStream_t stream);
hipError_t launch_softmax_bwd(const SoftmaxDesc& d, int dtype, hipStream_t stream);

// Fused attention forward (score, softmax and context in one kernel, no
// AS or AP in memory): bf16 storage, S a multiple of 128, head_dim 64 or
// 128, R dividing 128.
struct FusedDesc {
  int B = 0, nh = 0, S = 0, H = 0, D = 0, R = 128;
  int causal = 0;
  float scale = 1.f;
  const void* qkv = nullptr;   // [B*S][3H] bf16: Q | K | V column blocks
  const float* qkvc = nullptr; // [B][S/R][2][3H] propagated column checksums (K^c used)
  const float* vr = nullptr;   // [B*S][nh][2] propagated V^r (row checksums per head);
                               // carried through P V when given (CL check, CL^r)
  void* cl = nullptr;          // [B*S][H] bf16 output
  int check_as = 0, check_cl = 0;
  int recompute = 1;           // located score errors: recompute (else checksum fix)
  float e_rel = 0.f, tn_s = 0.f, tn_cl = 0.f, tc = 0.f;  // thresholds as compared
  const abft_fault* faults = nullptr;
  int n_faults = 0;
  abft_report* report = nullptr;
  // for the backward (may be null): per query the log2-scaled running max
  // and the sum of the online softmax [B][nh][S][2], and CL^r = A^r / l,
  // the propagated row checksums of CL [B*S][nh][2]
  float* stats = nullptr;
  float* clr = nullptr;
  // optional transposed bf16 image of CL^r [nh][4][B*S] (rows c1 hi, c1 lo,
  // c2 hi, c2 lo per head): the column strip of the dW^O GEMM
  uint16_t* clri = nullptr;
  // optional CL^c [B][S/R][2][H] (the column checksums of the stored,
  // checked CL over each R-query block) and its bf16 image [B][S/R][4][H]
  // (rows c1 hi, c1 lo, c2 hi, c2 lo): the output projection's strip
  float* clc = nullptr;
  uint16_t* clci = nullptr;
};
hipError_t launch_fused_fwd(const FusedDesc& d, hipStream_t stream);

// Fused backward core after a fused forward (no scores kept), in two
// passes that each recompute the scores from the softmax statistics: the
// query pass (dQ; it also leaves D = dCL . CL per query) and the key pass
// (dK and dV), which reads D. The row checksums over each head's dims
// (K^r in the query pass, Q^r and dCL^r in the key pass) are formed in the
// passes from the tiles they stage.
struct FusedBwdDesc {
  int B = 0, nh = 0, S = 0, H = 0, D = 0, R = 128;
  int causal = 0;
  float scale = 1.f;
  const void* qkv = nullptr;    // [B*S][3H] bf16: Q | K | V
  const float* qkvc = nullptr;  // [B][S/R][2][3H] propagated column checksums (Q^c, K^c, V^c)
  const float* dclc = nullptr;  // [B][S/R][2][H] propagated column checksums of dCL
  const void* cl = nullptr;     // [B*S][H] bf16, the forward's context
  const void* dcl = nullptr;    // [B*S][H] bf16
  const float* stats = nullptr; // [B][nh][S][2]: log2-scaled max and sum per query
  float* drow = nullptr;        // [B][nh][S]: D per query (query pass out, key pass in)
  void* dqkv = nullptr;         // out: [B*S][ld] bf16, dQ | dK | dV (head h at h D of each)
  int64_t ld = 0;
  int check = 0;                // run the checks
  int recompute = 1;            // located S / dP errors: recompute (else checksum fix)
  float e_rel = 0.f, tn_s = 0.f, tn = 0.f, tc = 0.f;
  const abft_fault* faults = nullptr;
  int n_faults = 0;
  abft_report* report = nullptr;
};
hipError_t launch_fused_bwd_q(const FusedBwdDesc& d, hipStream_t stream);
hipError_t launch_fused_bwd_kv(const FusedBwdDesc& d, hipStream_t stream);

// Checksum encoder (public encode_checksums) and standalone verifier.
hipError_t launch_encode(const void* A, int dtype, int64_t batch, int64_t rows, int64_t cols,
                         int64_t ld, int64_t batch_stride, int Rb, int Cb, float* col_chk,
                         float* row_chk, hipStream_t stream);
hipError_t launch_verify(void* C, int dtype, int64_t batch, int64_t rows, int64_t cols,
                         int64_t ld, int64_t batch_stride, int Rb, int Cb, float* col_chk,
                         float* row_chk, float tn, float tc, float e_rel, int op_tag,
                         abft_report* report, hipStream_t stream);
hipError_t launch_report_reset(abft_report* report, int capacity, bool set_capacity,
                               hipStream_t stream);

// Up to three encodes (each as launch_encode) and, when `reset` is given,
// the report's counters cleared as launch_report_reset(reset, 0, false)
// does; in one launch when all take the vector path with one slab width
// (else one launch each).
struct EncodeJob {
  const void* A = nullptr;
  int64_t batch = 0, rows = 0, cols = 0, ld = 0, batch_stride = 0;
  int Rb = 0, Cb = 0;
  float* col_chk = nullptr;
  float* row_chk = nullptr;
  int64_t ldcc = 0;  // elements between column-checksum rows (0: cols)
  // optional bf16 image of the column checksums (bf16 operands): per Rb-row
  // block four rows c1 hi, c1 lo, c2 hi, c2 lo of ldci elements, hi =
  // bf16(c), lo = bf16(c - hi)
  uint16_t* col_img = nullptr;
  int64_t ldci = 0;
  // optional bf16 image of the row checksums, transposed: per Cb-column
  // block four rows (c1 hi, c1 lo, c2 hi, c2 lo) over all batch x rows
  // rows of the operand, each ldri elements long
  uint16_t* row_img = nullptr;
  int64_t ldri = 0;
};
hipError_t launch_encode_jobs(const EncodeJob* jobs, int n, int dtype, abft_report* reset,
                              hipStream_t stream);

// Threshold as the storage dtype represents it (round to nearest even).
float stored_threshold(float t, int dtype);

}  // namespace abft
