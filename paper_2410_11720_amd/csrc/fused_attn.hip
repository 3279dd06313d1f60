// Fused protected attention, forward: the score, softmax and context steps
// of the layer (Sec. 2.1 Eq. 1-2) with the S_AS and S_CL checks of
// Sec. 4.4, in an online-softmax form that keeps neither the scores AS nor
// the probabilities AP in memory (an extension: the paper stores both).
//
// One workgroup per (batch, head, tile of 128 queries): four waves of 32
// queries (two workgroups per CU), or, protected at head dim 128, eight
// waves of 16 (one workgroup per CU; the registers of 32 queries spill
// there). Key tiles of 128 keys pass through LDS in order (causal: up to
// the diagonal tile), double-buffered where the LDS allows. Per key tile
// each wave computes
//   S^T = K Q^T on the matrix cores, keys as rows and queries as columns,
//     so a lane holds 32 keys of one query: the reductions over keys stay
//     in the lane and its three partners, and P^T feeds the next product
//     from registers;
//   AS^r = Q (K^c)^T from a strip of 16 extra key rows holding the
//     propagated K^c of the tile's R-key blocks as hi/lo bf16 rows;
//   the row check of every (query, R-key block) vector (sum against AS^r,
//     Sec. 2.3 rule); a flagged vector is located by EEC (Sec. 4.2) inside
//     the wave and its element recomputed from Q and K (or, with the root
//     check off, fixed from the checksums);
//   the online softmax (exp2 of log2(e)-scaled scores, running max and
//     per-lane partial sums);
//   O^T += V^T P^T and (A^r)^T += (V^r)^T P^T, both rescaled alike, so
//     A^r / l is the propagated row checksum of CL (V^r = X W^V r).
// After the last key tile CL = O / l is rounded, row-checked against
// A^r / l (located elements fixed from the checksum, Sec. 4.2) and stored.
// The column side of AS (AS^c = Q^c K^T) is not checked here: it would
// need a reduction across the 16 lanes of a query group per key. The fused
// form verifies Q, K and V at their projection in every mode, so the 1R
// and 1C patterns their errors would make cannot arise, and the rows
// locate the 0D pattern that remains.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "abft_internal.hpp"
#include "abft_device.hpp"
#include "direct_lds.hpp"

namespace abft {
namespace {

constexpr int FT = 128;   // queries per workgroup, keys per key tile

// x combined with the value of lane l ^ 16 (l ^ 32): the gfx950 lane-swap
// moves hand back both halves of the exchanged pair, so every lane gets
// the same result.
__device__ __forceinline__ float xsum16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xsum32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xmax16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xmax32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
// sum over the four 16-lane groups (the four lanes sharing lane % 16)
__device__ __forceinline__ float group4_sum(float x) { return xsum32(xsum16(x)); }

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  return uint32_t(f2bf(a)) | (uint32_t(f2bf(b)) << 16);
}
// the same in one packed conversion (the same rounding; used where the
// register allocation of the surrounding code allows it)
__device__ __forceinline__ uint32_t pack2v(float a, float b) {
  typedef float float2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const float2_t f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}
__device__ __forceinline__ float flip_f32(float x) {
  return __uint_as_float(__float_as_uint(x) ^ 0x40000000u);
}
__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Access to a kernel's descriptor, its only argument. With SEG, through
// the address of the kernel-argument segment, and refresh() makes that
// address opaque to the compiler, so fields read after it are loaded
// (scalar loads) where they are used instead of being held in scalar
// registers from an earlier read; without, plainly through the argument.
template <class Desc, bool SEG>
struct ArgRef {
  const Desc* p;
  __device__ explicit ArgRef(const Desc& d) : p(&d) {}
  __device__ void refresh() {}
  __device__ const Desc* operator->() const { return p; }
};
#if defined(__HIP_DEVICE_COMPILE__)  // the host pass emits no device code
template <class Desc>
struct ArgRef<Desc, true> {
  decltype(__builtin_amdgcn_kernarg_segment_ptr()) p;
  __device__ explicit ArgRef(const Desc&) : p(__builtin_amdgcn_kernarg_segment_ptr()) {}
  __device__ void refresh() { asm volatile("" : "+s"(p)); }
  __device__ const Desc* operator->() const { return (const Desc*)p; }
};
#endif

// Sums over a float vector scr[0..n) (n <= 128) in LDS across the wave:
// lane l holds elements l and l + 64 (zero past n); every lane gets the
// totals.
struct WaveVec {
  float x0, x1;
  bool in0, in1;
  __device__ WaveVec(const float* scr, int n, int lane)
      : in0(lane < n), in1(lane + 64 < n) {
    x0 = in0 ? scr[lane] : 0.f;
    x1 = in1 ? scr[lane + 64] : 0.f;
  }
};

// EEC-ABFT location (Sec. 4.2) of a flagged vector, wave-parallel: the
// same decisions as the one-lane form in abft_device.hpp (sums in another
// order: both are fp32 approximations of the exact sums), the candidates
// counted by ballots, the located candidate the last one.
__device__ EecResult eec_wave(const WaveVec& v, int lane, int n, float c1, float c2, float e_rel,
                              float tn) {
  const float r1 = group_sum<64>(v.x0 + v.x1);
  const float r2 = group_sum<64>(fmaf(float(lane + 1), v.x0, float(lane + 65) * v.x1));
  const float sa = group_sum<64>((is_finite(v.x0) ? fabsf(v.x0) : 0.f) +
                                 (is_finite(v.x1) ? fabsf(v.x1) : 0.f));
  const float d1 = c1 - r1, d2 = c2 - r2;
  EecResult res{EEC_CLEAN, -1, d1};
  if (!flagged(d1, sa, e_rel)) return res;
  const int mode = is_finite(d1) ? 1 : (is_inf(d1) ? 2 : 3);
  const bool any_inf = mode == 2, any_nonfin = mode == 3;
  auto cand = [&](float x, bool in) {
    const bool fin = is_finite(x);
    return in && ((fin && fabsf(x) >= tn) || (any_inf && is_inf(x)) || (any_nonfin && !fin));
  };
  const uint64_t b0 = __ballot(cand(v.x0, v.in0)), b1 = __ballot(cand(v.x1, v.in1));
  const int cnt = __popcll(b0) + __popcll(b1);
  const int idx = b1 ? 127 - __clzll(b1) : (b0 ? 63 - __clzll(b0) : -1);
  res.status = EEC_PROPAGATED;
  if (cnt >= 2) return res;
  if (mode == 1) {
    if (cnt == 1) {
      if (is_finite(d2)) {
        const float q = d2 / d1;
        if (!(fabsf(q - float(idx + 1)) < 0.25f)) return res;
      }
      res.status = EEC_LOCATED;
      res.index = idx;
      return res;
    }
    if (!is_finite(d2)) return res;
    const float q = d2 / d1;
    if (!(q >= 0.5f && q < float(n) + 0.5f)) return res;
    const float qi = rintf(q);
    if (!(fabsf(q - qi) < 0.25f)) return res;
    res.status = EEC_LOCATED;
    res.index = int(qi) - 1;
    return res;
  }
  if (cnt == 1) {
    res.status = EEC_LOCATED;
    res.index = idx;
  }
  return res;
}

// The detection rule on a vector (sum against c1, bound from the
// magnitudes), wave-parallel.
__device__ bool flagged_wave(const WaveVec& v, float c1, float e_rel) {
  const float r1 = group_sum<64>(v.x0 + v.x1);
  const float sa = group_sum<64>(fabsf(v.x0) + fabsf(v.x1));
  return flagged(c1 - r1, sa, e_rel);
}

// Fixing a flagged score vector gathered in scr[0..n) (Sec. 4.2), in up to
// three steps, by the whole wave (every lane calls them). score_locate
// locates by EEC; a located element is fixed from the checksums (DELTA or
// RECONSTRUCT) unless recompute is set, the event recorded at (row, col)
// when tr, else (col, row), and an unfixable vector reported; scr[n] takes
// the located index (or -1), scr[n + 1] the new value. With recompute, a
// located element is left to score_dot, which forms the dot product of row
// `col` of A and row `rowbase + index` of Bm (length d <= 128) across the
// lanes, then score_close stores it, records the event and reports a vector
// that is still flagged. Lane 0 writes scr[n], scr[n + 1] and the events.
__device__ __noinline__ void score_locate(float* scr, int n, float v1, float v2, float e_rel,
                                          float tn, float tc, int recompute, abft_report* report,
                                          int op, int b, int h, int col, int rowbase, bool tr,
                                          int lane) {
  const WaveVec v(scr, n, lane);
  const EecResult res = eec_wave(v, lane, n, v1, v2, e_rel, tn);
  int idx = -1;
  float nv = 0.f;
  bool still = false;
  if (res.status == EEC_LOCATED) {
    idx = res.index;
    const float old = scr[idx];
    if (recompute) {  // the rest after score_dot
      if (lane == 0) {
        scr[n] = __int_as_float(idx);
        scr[n + 1] = old;
      }
      return;
    }
    int action;
    if (is_finite(res.d1) && fabsf(res.d1) <= tc) {
      action = ABFT_ACT_DELTA;
      nv = old + res.d1;
    } else {
      action = ABFT_ACT_RECONSTRUCT;
      const float rest = (lane == idx ? 0.f : v.x0) + (lane + 64 == idx ? 0.f : v.x1);
      nv = v1 - group_sum<64>(rest);
    }
    const int row = rowbase + idx;
    if (lane == 0)
      record_event(report, op, b, h, tr ? row : col, tr ? col : row, classify(old, tn), action,
                   old);
    WaveVec w = v;  // the vector with the fix
    if (lane == idx) w.x0 = nv;
    if (lane + 64 == idx) w.x1 = nv;
    still = flagged_wave(w, v1, e_rel);
    if (lane == 0) scr[idx] = nv;
  } else if (res.status != EEC_CLEAN) {
    still = flagged_wave(v, v1, e_rel);
  }
  if (lane == 0) {
    if (still)
      record_event(report, op, b, h, tr ? rowbase : col, tr ? col : rowbase, ABFT_KIND_NONE,
                   ABFT_ACT_UNCORRECTABLE, 0.f);
    scr[n] = __int_as_float(idx);
    scr[n + 1] = nv;
  }
}
__device__ __noinline__ float score_dot(const bf16_t* A, const bf16_t* Bm, int64_t lda,
                                           int64_t ldb, int col, int row, int d, int lane) {
  float acc = 0.f;
  for (int dd = lane; dd < d; dd += 64)
    acc = fmaf(bf2f(A[int64_t(col) * lda + dd]), bf2f(Bm[int64_t(row) * ldb + dd]), acc);
  return group_sum<64>(acc);
}
__device__ __noinline__ void score_close(float* scr, int n, float nv, float v1, float e_rel,
                                         float tn, abft_report* report, int op, int b, int h,
                                         int col, int rowbase, bool tr, int lane) {
  const int idx = __float_as_int(scr[n]);
  const int row = rowbase + idx;
  const float old = scr[idx];
  WaveVec w(scr, n, lane);
  if (lane == idx) w.x0 = nv;
  if (lane + 64 == idx) w.x1 = nv;
  const bool still = flagged_wave(w, v1, e_rel);
  if (lane == 0) {
    scr[idx] = nv;
    record_event(report, op, b, h, tr ? row : col, tr ? col : row, classify(old, tn),
                 ABFT_ACT_RECOMPUTE, old);
    if (still)
      record_event(report, op, b, h, tr ? rowbase : col, tr ? col : rowbase, ABFT_KIND_NONE,
                   ABFT_ACT_UNCORRECTABLE, 0.f);
    scr[n + 1] = nv;
  }
}

// A flagged row vector of an output (CL in the forward; dQ, dK, dV in the
// backward passes) gathered in scr[0..n) (n <= 128), by the whole wave:
// located by EEC and fixed from its checksums (DELTA or RECONSTRUCT, the
// new value rounded to bf16 as stored), the event recorded at (e, index),
// an unfixable vector reported; scr[n] takes the located index (or -1),
// scr[n + 1] the new value (lane 0 writes them and the events).
__device__ __noinline__ void grad_fix(float* scr, int n, float v1, float v2, float e_rel, float tn,
                                      float tc, abft_report* report, int op, int b, int h, int e,
                                      int lane) {
  const WaveVec v(scr, n, lane);
  const EecResult res = eec_wave(v, lane, n, v1, v2, e_rel, tn);
  int idx = -1;
  float nv = 0.f;
  bool still = false;
  if (res.status == EEC_LOCATED) {
    idx = res.index;
    const float old = scr[idx];
    int action;
    if (is_finite(res.d1) && fabsf(res.d1) <= tc) {
      action = ABFT_ACT_DELTA;
      nv = old + res.d1;
    } else {
      action = ABFT_ACT_RECONSTRUCT;
      const float rest = (lane == idx ? 0.f : v.x0) + (lane + 64 == idx ? 0.f : v.x1);
      nv = v1 - group_sum<64>(rest);
    }
    nv = bf2f(f2bf(nv));
    if (lane == 0) record_event(report, op, b, h, e, idx, classify(old, tn), action, old);
    WaveVec w = v;
    if (lane == idx) w.x0 = nv;
    if (lane + 64 == idx) w.x1 = nv;
    still = flagged_wave(w, v1, e_rel);
    if (lane == 0) scr[idx] = nv;
  } else if (res.status != EEC_CLEAN) {
    still = flagged_wave(v, v1, e_rel);
  }
  if (lane == 0) {
    if (still) record_event(report, op, b, h, e, 0, ABFT_KIND_NONE, ABFT_ACT_UNCORRECTABLE, 0.f);
    scr[n] = __int_as_float(idx);
    scr[n + 1] = nv;
  }
}

// Whether an injected fault (test-only) of an op in mask targets head
// (b, h) of a batch element: read once per workgroup, so that the
// workgroups no fault reaches skip the per-tile injection code (each of its
// passes reads the fault list from memory).
__device__ __forceinline__ bool faults_at(const abft_fault* f, int n, int b, int h,
                                          uint32_t mask) {
  bool any = false;
  for (int i = 0; i < n; ++i) {
    const abft_fault ft = f[i];
    any |= ft.op >= 0 && ft.op < 32 && ((mask >> ft.op) & 1u) && ft.b == b && ft.h == h;
  }
  return any;
}

template <int D, bool PROT>
struct FusedAttn {
  // 16-query blocks per wave: one for the protected kernel at head dim 128
  // (two would spill), else two (fewer LDS reads per MFMA)
  static constexpr int QB = D == 128 && PROT ? 1 : 2;
  static constexpr int NTH = 64 * (FT / (16 * QB));   // threads per workgroup
  static constexpr int NW = NTH / 64;
  // LDS stages of key tiles: two, except where two workgroups per CU leave
  // room for one (head dim 128, four waves)
  static constexpr int NSTAGE = D == 64 || QB == 1 ? 2 : 1;
  static constexpr int KH = D / 64;    // 64-wide halves of the head dim (K images)
  static constexpr int KS = D / 32;    // k steps of the score product
  static constexpr int DB = D / 16;    // 16-row blocks of O^T
  using DK = Direct<true, FT, NTH>;    // K half [128 keys][64 dims], swizzled
  using DV = Direct<false, D, NTH>;    // V image [64 keys][D dims], swizzled
  static constexpr int K_BYTES = KH * DK::BYTES;
  static constexpr int V_BYTES = 2 * DV::BYTES;
  static constexpr int KCL = D + 8;    // K^c strip row (elements), padded
  static constexpr int KC_BYTES = PROT ? 16 * KCL * 2 : 0;
  static constexpr int VR_BYTES = PROT ? FT * 16 * 2 : 0;
  static constexpr int STAGE_BYTES = K_BYTES + V_BYTES + KC_BYTES + VR_BYTES;
  static constexpr int SCR = 160;      // floats of rare-path scratch per wave
  static constexpr int LDS_BYTES = NSTAGE * STAGE_BYTES + (PROT ? NW * SCR * 4 : 0);
  static_assert(LDS_BYTES <= (QB == 2 ? 80 : 160) * 1024, "two (one) workgroups per CU");

  // V^T operand fragment for keys {kb + 4g + v, kb + 16 + 4g + v} (g = lane
  // group, v = 0..3), rows (dims) rb + lane % 16: the key order of the P^T
  // fragment a lane assembles from its S^T accumulators.
  // (transposing reads: valid after lds_wait_all(), through tr_join(); head
  // dim 128 and the unprotected kernel keep the compiler's intrinsic, which
  // measured faster there: its own waits cost less than the registers and
  // coarser waits of the assembly form)
  __device__ static __forceinline__ TrPair vt_frag(const char* st, int rb, int kb, int lane) {
    const int s = lane & 15, g = lane >> 4;
    const int k1 = kb + 4 * g + (s >> 2), k2 = k1 + 16;
    const int m = rb + 4 * (s & 3);
    const int c = m >> 3, off = (m & 7) * 2;
    const char* p0 = st + k1 * (D * 2) + ((c ^ (2 * (k1 & 3))) << 4) + off;
    const char* p1 = st + k2 * (D * 2) + ((c ^ (2 * (k2 & 3))) << 4) + off;
    if constexpr (D == 64 && PROT) return tr_pair(p0, p1);
    else return tr_pair_intrinsic(p0, p1);
  }
  // (V^r)^T fragment from the plain [128 keys][16] strip, same key order
  __device__ static __forceinline__ TrPair vr_frag(const bf16_t* vrs, int kb, int lane) {
    const int s = lane & 15, g = lane >> 4;
    const int k1 = kb + 4 * g + (s >> 2), k2 = k1 + 16;
    const int m = 4 * (s & 3);
    if constexpr (D == 64 && PROT) return tr_pair(vrs + k1 * 16 + m, vrs + k2 * 16 + m);
    else return tr_pair_intrinsic(vrs + k1 * 16 + m, vrs + k2 * 16 + m);
  }

  __device__ static void run(const FusedDesc& fd, char* smem) {
    ArgRef<FusedDesc, D == 64> arg(fd);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lq = lane & 15, g = lane >> 4;
    const int nqt = arg->S / FT, nbh = arg->B * arg->nh;
    const int z = blockIdx.x % nbh;
    // causal: the heaviest query tiles (most key tiles) start first
    const int qt = arg->causal ? nqt - 1 - int(blockIdx.x) / nbh : int(blockIdx.x) / nbh;
    const int b = z / arg->nh, h = z % arg->nh;
    const int q0 = qt * FT, qw = q0 + wave * 16 * QB;
    const int S = arg->S, H = arg->H;
    const int64_t ld = 3 * int64_t(H);
    const bf16_t* base = static_cast<const bf16_t*>(arg->qkv) + int64_t(b) * S * ld;
    const bf16_t* Qp = base + h * D;
    const bf16_t* Kp = base + H + h * D;
    const bf16_t* Vp = base + 2 * H + h * D;
    const int nkt = arg->causal ? qt + 1 : nqt;
    const int R = arg->R, NB = FT / R;                  // checksum blocks per key tile
    const int lg_jpb = __builtin_ctz(R / 16);         // 16-key groups per block (log2)
    const float sl2 = arg->scale * 1.4426950408889634f;
    const bool wf = arg->n_faults > 0 &&
                    faults_at(arg->faults, arg->n_faults, b, h,
                              (1u << ABFT_OP_AS) | (1u << ABFT_OP_CL));

    // Q as the B operand of S^T: query qw + 16 qb + lane % 16, dims 32 kk + 8 g..
    bf16x8 qf[QB][KS];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        qf[qb][kk] = *reinterpret_cast<const bf16x8*>(Qp + int64_t(qw + 16 * qb + lq) * ld +
                                                        32 * kk + 8 * g);

    // checksum strip registers (loaded with a tile, written to LDS when it lands)
    float kcv[4] = {0.f, 0.f, 0.f, 0.f};
    float vrv = 0.f;
    auto issue = [&](int kt, int st) {
      char* sb = smem + st * STAGE_BYTES;
      const int key0 = kt * FT;
#pragma unroll
      for (int hf = 0; hf < KH; ++hf) DK::issue(Kp, ld, key0, S, hf * 64, sb + hf * DK::BYTES, wave, lane);
#pragma unroll
      for (int im = 0; im < 2; ++im)
        DV::issue(Vp, ld, 0, D, key0 + 64 * im, sb + K_BYTES + im * DV::BYTES, wave, lane);
      if constexpr (PROT) {
        if (arg->check_as) {
          const int nqR = S / R;
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            const int e = tid + p * NTH;
            const bool ok = e < NB * 2 * D;
            const int ee = ok ? e : 0;
            const int blk = ee / (2 * D), c = (ee / D) & 1, dd = ee % D;
            // (used by commit only where e is in range: no select here, which
            // would wait for the load, and with it for the tile's loads)
            kcv[p] = arg->qkvc[((int64_t(b) * nqR + key0 / R + blk) * 2 + c) * ld + H + h * D + dd];
          }
        }
        // threads 0..255: the tile's 128 keys x (c1, c2)
        if (arg->vr != nullptr && tid < 2 * FT)
          vrv = arg->vr[((int64_t(b) * S + key0 + (tid >> 1)) * arg->nh + h) * 2 + (tid & 1)];
      }
    };
    auto commit = [&](int st) {
      if constexpr (PROT) {
        char* sb = smem + st * STAGE_BYTES;
        if (arg->check_as) {
          bf16_t* kcs = reinterpret_cast<bf16_t*>(sb + K_BYTES + V_BYTES);
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            const int e = tid + p * NTH;
            if (e < NB * 2 * D) {
              const int blk = e / (2 * D), c = (e / D) & 1, dd = e % D;
              const bf16_t hi = f2bf(kcv[p]);
              const bf16_t lo = f2bf(kcv[p] - bf2f(hi));
              kcs[(4 * blk + 2 * c) * KCL + dd] = hi;
              kcs[(4 * blk + 2 * c + 1) * KCL + dd] = lo;
            }
          }
        }
        if (arg->vr != nullptr && tid < 2 * FT) {
          bf16_t* vrs = reinterpret_cast<bf16_t*>(sb + K_BYTES + V_BYTES + KC_BYTES);
          const bf16_t hi = f2bf(vrv);
          const bf16_t lo = f2bf(vrv - bf2f(hi));
          vrs[(tid >> 1) * 16 + 2 * (tid & 1)] = hi;
          vrs[(tid >> 1) * 16 + 2 * (tid & 1) + 1] = lo;
        }
      }
    };
    if constexpr (PROT) {  // the V^r strip columns past the four used ones stay zero
      for (int st = 0; st < NSTAGE; ++st) {
        bf16_t* vrs = reinterpret_cast<bf16_t*>(smem + st * STAGE_BYTES + K_BYTES + V_BYTES + KC_BYTES);
        for (int e = tid; e < FT * 12; e += NTH) vrs[(e / 12) * 16 + 4 + e % 12] = 0;
      }
    }

    floatx4 o[DB][QB], vra[QB];
    float m[QB], l[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db][qb] = floatx4{0.f, 0.f, 0.f, 0.f};
      vra[qb] = floatx4{0.f, 0.f, 0.f, 0.f};
      m[qb] = -INFINITY;
      l[qb] = 0.f;
    }
    float* scr = reinterpret_cast<float*>(smem + NSTAGE * STAGE_BYTES) + wave * SCR;

    if (NSTAGE == 2) issue(0, 0);
    for (int kt = 0; kt < nkt; ++kt) {
      // with head dim 64 the descriptor's fields are loaded per key tile
      // (fewer scalar registers held across the loop); with 128 that costs
      // more vector registers than it saves
      arg.refresh();
      const int st = NSTAGE == 2 ? (kt & 1) : 0;
      if (NSTAGE == 1) issue(kt, 0);
      wait_vmcnt<0>();
      commit(st);
      __syncthreads();  // tile kt visible; every wave is done with tile kt - 1
      if (NSTAGE == 2 && kt + 1 < nkt) issue(kt + 1, st ^ 1);
      const char* sb = smem + st * STAGE_BYTES;
      const int key0 = kt * FT;

      // S^T (and AS^r from the strip)
      floatx4 s[8][QB], ks[QB];
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) s[j][qb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) ks[qb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const char* sk = sb + (kk >> 1) * DK::BYTES;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const bf16x8 kf = DK::frag(sk, 16 * j, (kk & 1) * 32, lane);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            s[j][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[qb][kk], s[j][qb], 0, 0, 0);
        }
        if constexpr (PROT) {
          if (arg->check_as) {
            const bf16_t* kcs = reinterpret_cast<const bf16_t*>(sb + K_BYTES + V_BYTES);
            const bf16x8 sf = *reinterpret_cast<const bf16x8*>(kcs + lq * KCL + 32 * kk + 8 * g);
#pragma unroll
            for (int qb = 0; qb < QB; ++qb)
              ks[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sf, qf[qb][kk], ks[qb], 0, 0, 0);
          }
        }
      }

      // injected score faults (test-only), on the unrounded scores
      if (wf) {
        for (int f = 0; f < arg->n_faults; ++f) {
          const abft_fault ft = arg->faults[f];
          if (ft.op != ABFT_OP_AS || ft.b != b || ft.h != h) continue;
          const int qi = ft.row - qw, ki = ft.col - key0;
          if (qi < 0 || qi >= 16 * QB || ki < 0 || ki >= FT) continue;
          const int oq = qi >> 4, olane = (qi & 15) + 16 * ((ki & 15) >> 2);
#pragma unroll
          for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int qb = 0; qb < QB; ++qb)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (lane == olane && qb == oq && j == (ki >> 4) && r == (ki & 3))
                  s[j][qb][r] = ft.mode == ABFT_FAULT_FLIP ? flip_f32(s[j][qb][r]) : ft.value;
        }
      }

      // row check of S per (query, R-key block)
      if constexpr (PROT) {
        if (arg->check_as) {
          uint64_t fmask[QB];
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) {
            // block sums of the values and, only when a vector needs them,
            // of the magnitudes (2, 4 or 8 groups of 16 keys, reduced over
            // the 4 lanes): as |sum| <= sum of magnitudes, a vector whose
            // sum is within e_rel |sum| (shrunk by 0.1%, far beyond the
            // rounding of either sum) of its checksum passes the rule
            // whatever its magnitude sum
            auto block_sums = [&](auto mag) {
              float sj[8];
#pragma unroll
              for (int j = 0; j < 8; ++j) {
                if constexpr (decltype(mag)::value)
                  sj[j] = (fabsf(s[j][qb][0]) + fabsf(s[j][qb][1])) +
                          (fabsf(s[j][qb][2]) + fabsf(s[j][qb][3]));
                else
                  sj[j] = (s[j][qb][0] + s[j][qb][1]) + (s[j][qb][2] + s[j][qb][3]);
              }
              float r1[4];
#pragma unroll
              for (int i = 0; i < 4; ++i) r1[i] = sj[2 * i] + sj[2 * i + 1];
              if (lg_jpb >= 2) {
                r1[0] += r1[1];
                r1[1] = r1[2] + r1[3];
              }
              if (lg_jpb >= 3) r1[0] += r1[1];
              float mine = 0.f;
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                if (i < NB) {
                  const float t1 = group4_sum(r1[i]);
                  if (g == i) mine = t1;
                }
              }
              return mine;
            };
            const float mine1 = block_sums(std::false_type{});
            const float d = ks[qb][0] + ks[qb][1] - mine1;
            const bool clear =
                g >= NB || (is_finite(d) && fabsf(d) <= arg->e_rel * fabsf(mine1) * 0.999f);
            float minea = INFINITY;
            if (__ballot(!clear) != 0) minea = block_sums(std::true_type{});
            const float c1 = ks[qb][0] + ks[qb][1];
            const bool fl = g < NB && flagged(c1 - mine1, minea, arg->e_rel);
            fmask[qb] = __ballot(fl);
          }
          uint64_t any = 0;
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) any |= fmask[qb];
          if (any) {  // rare: locate and correct inside the wave
            // the tile's scores wait in private memory (indexed at run time,
            // so they stay there): no score register is live while the
            // flagged vectors are corrected
            float sm[QB][8][4];
#pragma unroll
            for (int qb = 0; qb < QB; ++qb)
#pragma unroll
              for (int j = 0; j < 8; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) sm[qb][j][r] = s[j][qb][r];
            const int jpb = 1 << lg_jpb;
            for (int qb = 0; qb < QB; ++qb) {
              uint64_t mask = fmask[qb];
              const float cs1 = ks[qb][0] + ks[qb][1], cs2 = ks[qb][2] + ks[qb][3];
              while (mask) {
                const int L = __builtin_ctzll(mask);
                mask &= mask - 1;
                const int vq = L & 15, vb = L >> 4;    // query lane, key block
                // gather the vector S[q][block vb] into the scratch
                if (lq == vq) {
                  for (int jj = 0; jj < jpb; ++jj) {
                    const int j = vb * jpb + jj;
#pragma unroll
                    for (int r = 0; r < 4; ++r) scr[16 * jj + 4 * g + r] = sm[qb][j][r];
                  }
                }
                const float v1 = __shfl(cs1, L, 64);
                const float v2 = __shfl(cs2, L, 64);
                wave_sync_lds();
                score_locate(scr, R, v1, v2, arg->e_rel, arg->tn_s, arg->tc, arg->recompute,
                             arg->report, ABFT_OP_AS, b, h, qw + 16 * qb + vq, key0 + vb * R,
                             false, lane);
                wave_sync_lds();
                if (arg->recompute && __float_as_int(scr[R]) >= 0) {
                  const float nv = score_dot(Qp, Kp, ld, ld, qw + 16 * qb + vq,
                                             key0 + vb * R + __float_as_int(scr[R]), D, lane);
                  score_close(scr, R, nv, v1, arg->e_rel, arg->tn_s, arg->report, ABFT_OP_AS,
                              b, h, qw + 16 * qb + vq, key0 + vb * R, false, lane);
                }
                wave_sync_lds();
                const int idx = __float_as_int(scr[R]);
                const float nv = scr[R + 1];
                if (idx >= 0) {
                  const int kl = vb * R + idx;
                  if (lane == vq + 16 * ((kl & 15) >> 2)) sm[qb][kl >> 4][kl & 3] = nv;
                }
                wave_sync_lds();
              }
            }
#pragma unroll
            for (int qb = 0; qb < QB; ++qb)
#pragma unroll
              for (int j = 0; j < 8; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) s[j][qb][r] = sm[qb][j][r];
          }
        }
      }

      // online softmax, then O^T += V^T P^T (and the V^r rows). The
      // running max is kept in the log2-scaled domain; the tile's max is
      // taken over the raw scores and scaled once (the scale is positive,
      // so the result is the same), and each probability is exp2 of one
      // fused multiply-add.
      if (arg->causal && kt == qt) {
        // the diagonal tile's masked scores
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (key0 + 16 * j + 4 * g + r > qw + 16 * qb + lq) s[j][qb][r] = -INFINITY;
      }
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) mx = fmaxf(mx, s[j][qb][r]);
        mx = xmax32(xmax16(mx)) * sl2;
        const float mn = fmaxf(m[qb], mx);
        const float alpha = __builtin_amdgcn_exp2f(m[qb] - mn);
        m[qb] = mn;
        float ls = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float p = __builtin_amdgcn_exp2f(fmaf(s[j][qb][r], sl2, -mn));
            s[j][qb][r] = p;
            ls += p;
          }
        l[qb] = l[qb] * alpha + ls;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db][qb] *= alpha;
        vra[qb] *= alpha;
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const char* sv = sb + K_BYTES + (t >> 1) * DV::BYTES;
        // the first V^T read goes out before P is packed; each later one
        // before the MFMAs of the previous (one read pair in flight)
        TrPair cur = vt_frag(sv, 0, (t & 1) * 32, lane);
        bf16x8 pf[QB];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          const uint4 u = {pack2v(s[2 * t][qb][0], s[2 * t][qb][1]),
                           pack2v(s[2 * t][qb][2], s[2 * t][qb][3]),
                           pack2v(s[2 * t + 1][qb][0], s[2 * t + 1][qb][1]),
                           pack2v(s[2 * t + 1][qb][2], s[2 * t + 1][qb][3])};
          pf[qb] = __builtin_bit_cast(bf16x8, u);
        }
        const bool with_vr = PROT && arg->vr != nullptr;
        const bf16_t* vrs = reinterpret_cast<const bf16_t*>(sb + K_BYTES + V_BYTES + KC_BYTES);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          // (head dim 128: no read ahead, for registers)
          constexpr bool AHEAD = D == 64 && PROT;
          TrPair nxt = cur;
          bool more = AHEAD;
          if (!AHEAD) {
            if (db > 0) cur = vt_frag(sv, 16 * db, (t & 1) * 32, lane);
          } else if (db + 1 < DB) {
            nxt = vt_frag(sv, 16 * (db + 1), (t & 1) * 32, lane);
          } else if (with_vr) {
            nxt = vr_frag(vrs, 32 * t, lane);
          } else {
            more = false;
          }
          if (more) lds_wait_but2();
          else lds_wait_all();
          const bf16x8 vf = tr_join(cur);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            o[db][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[qb], o[db][qb], 0, 0, 0);
          cur = nxt;
        }
        if (with_vr && !(D == 64 && PROT)) cur = vr_frag(vrs, 32 * t, lane);
        if (with_vr) {
          lds_wait_all();
          const bf16x8 rf = tr_join(cur);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            vra[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rf, pf[qb], vra[qb], 0, 0, 0);
        }
      }
      if (NSTAGE == 1) __syncthreads();  // the one stage is reloaded next
    }

    // CL = O / l: round, check against A^r / l, store
    bf16_t* CLp = static_cast<bf16_t*>(arg->cl) + int64_t(b) * S * H + h * D;
    // CL^c of the stored CL (given clc): the lane's sums over its queries of
    // each of its dims (plain and weighted by the query's place in its
    // R-query block, from 1)
    float cs1[DB][4], cs2[DB][4];
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 4; ++r) cs1[db][r] = cs2[db][r] = 0.f;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int q = qw + 16 * qb + lq;
      const float lsum = group4_sum(l[qb]);
      const float inv = 1.f / lsum;
      if (arg->stats != nullptr && g == 0) {
        float* st = arg->stats + ((int64_t(b) * arg->nh + h) * S + q) * 2;
        st[0] = m[qb];
        st[1] = lsum;
      }
      if constexpr (PROT) {
        if (arg->vr != nullptr && arg->clr != nullptr && g == 0) {
          float* cr = arg->clr + ((int64_t(b) * S + q) * arg->nh + h) * 2;
          const float c1 = (vra[qb][0] + vra[qb][1]) * inv, c2 = (vra[qb][2] + vra[qb][3]) * inv;
          cr[0] = c1;
          cr[1] = c2;
          if (arg->clri != nullptr) {  // 16 consecutive queries per store
            const int64_t T = int64_t(arg->B) * S;
            bf16_t* ip = reinterpret_cast<bf16_t*>(arg->clri) + int64_t(h) * 4 * T + int64_t(b) * S + q;
            const bf16_t h1 = f2bf(c1), h2 = f2bf(c2);
            ip[0] = h1;
            ip[T] = f2bf(c1 - bf2f(h1));
            ip[2 * T] = h2;
            ip[3 * T] = f2bf(c2 - bf2f(h2));
          }
        }
      }
      float ov[DB][4];
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 4; ++r) ov[db][r] = bf2f(f2bf(o[db][qb][r] * inv));
      if (wf) {
        for (int f = 0; f < arg->n_faults; ++f) {
          const abft_fault ft = arg->faults[f];
          if (ft.op != ABFT_OP_CL || ft.b != b || ft.h != h || ft.row != q) continue;
          const int dd = ft.col;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (dd == 16 * db + 4 * g + r)
                ov[db][r] = ft.mode == ABFT_FAULT_FLIP ? bf2f(flip_exponent_msb(f2bf(ov[db][r])))
                                                       : bf2f(f2bf(ft.value));
        }
      }
      if constexpr (PROT) {
        if (arg->check_cl) {
          // the four lanes of the query take its checksums from lane group 0
          const float c1 = __shfl((vra[qb][0] + vra[qb][1]) * inv, lq, 64);
          const float c2 = __shfl((vra[qb][2] + vra[qb][3]) * inv, lq, 64);
          float r1 = 0.f, ra = 0.f;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              r1 += ov[db][r];
              ra += fabsf(ov[db][r]);
            }
          r1 = group4_sum(r1);
          ra = group4_sum(ra);
          uint64_t mask = __ballot(g == 0 && flagged(c1 - r1, ra, arg->e_rel));
          while (mask) {
            const int L = __builtin_ctzll(mask);
            mask &= mask - 1;
            if (lq == L) {
#pragma unroll
              for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int r = 0; r < 4; ++r) scr[16 * db + 4 * g + r] = ov[db][r];
            }
            const float v1 = __shfl(c1, L, 64), v2 = __shfl(c2, L, 64);
            wave_sync_lds();
            grad_fix(scr, D, v1, v2, arg->e_rel, arg->tn_cl, arg->tc, arg->report, ABFT_OP_CL, b,
                     h, qw + 16 * qb + L, lane);
            wave_sync_lds();
            const int idx = __float_as_int(scr[D]);
            const float nv = scr[D + 1];
            if (idx >= 0 && lq == L) {
#pragma unroll
              for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  if (idx == 16 * db + 4 * g + r) ov[db][r] = nv;
            }
            wave_sync_lds();
          }
        }
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const uint2 w = {pack2(ov[db][0], ov[db][1]), pack2(ov[db][2], ov[db][3])};
        *reinterpret_cast<uint2*>(CLp + int64_t(q) * H + 16 * db + 4 * g) = w;
      }
      if constexpr (PROT) {
        const float wq = float((q - q0) % arg->R + 1);
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float x = bf2f(f2bf(ov[db][r]));  // as stored
            cs1[db][r] += x;
            cs2[db][r] = fmaf(wq, x, cs2[db][r]);
          }
      }
    }
    if constexpr (PROT) {
      if (arg->clc != nullptr) {
        // sums over the wave's 16 query lanes (one DPP row per lane
        // group), then over the waves of each R-query block through LDS
        // (the stages are free once every wave is past the key loop), in
        // a fixed order
        __syncthreads();
        float* part = reinterpret_cast<float*>(smem);  // [NW][2][D]
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float t1 = group_sum<16>(cs1[db][r]), t2 = group_sum<16>(cs2[db][r]);
            if (lq == 0) {
              part[(wave * 2) * D + 16 * db + 4 * g + r] = t1;
              part[(wave * 2 + 1) * D + 16 * db + 4 * g + r] = t2;
            }
          }
        __syncthreads();
        const int R = arg->R, NBq = FT / R, wpb = NW / NBq;  // waves per R-query block
        const int nqR = S / R;
        for (int e = tid; e < NBq * 2 * D; e += NTH) {
          const int blk = e / (2 * D), c = (e / D) & 1, d = e % D;
          float v = 0.f;
          for (int w = blk * wpb; w < (blk + 1) * wpb; ++w) v += part[(w * 2 + c) * D + d];
          const int64_t row = int64_t(b) * nqR + q0 / R + blk;
          arg->clc[(row * 2 + c) * H + h * D + d] = v;
          if (arg->clci != nullptr) {
            const bf16_t hi = f2bf(v);
            bf16_t* ip = reinterpret_cast<bf16_t*>(arg->clci) + (row * 4 + 2 * c) * H + h * D + d;
            ip[0] = hi;
            ip[H] = f2bf(v - bf2f(hi));
          }
        }
      }
    }
  }
};

// Fused backward core (after a fused forward, which keeps no scores), in
// two passes that each recompute the scores from the forward's softmax
// statistics (no score-shaped tensor is read or written):
//  - the query pass, per (batch, head, tile of 128 queries), each wave
//    owning 32 queries and the key tiles passing through LDS: S^T = K Q^T
//    row-checked per (query, R-key block) against Q (K^c)^T, P from the
//    statistics, dP^T = V dCL^T row-checked against dCL (V^c)^T,
//    dS = scale P (dP - D) with D = dCL . CL (left in memory for the key
//    pass), dQ^T += K^T dS^T with (dQ^r)^T += (K^r)^T dS^T; dQ is rounded,
//    row-checked (a located element fixed from the checksum) and stored;
//  - the key pass, per (batch, head, tile of 128 keys), each wave owning 32
//    keys and the query tiles passing through LDS: S = Q K^T column-checked
//    per (R-query block, key) against (Q^c) K^T, P, dV^T += dCL^T P with
//    (dV^r)^T += (dCL^r)^T P, dP = dCL V^T column-checked against
//    (dCL^c) V^T, dS, dK^T += Q^T dS with (dK^r)^T += (Q^r)^T dS; dK and dV
//    are rounded, row-checked and stored.
// A workgroup of eight waves (two per SIMD) owns 128 columns; each wave
// works on a 128 x 16 score tile, the 128-long side along a lane's
// registers and lane groups, so its checks and the packing of P and dS into
// the next product's operand stay inside the wave; the two passes differ in
// which entity (query or key) is the 16-wide side. The located-element
// work of the checks runs out of line (it is rare and would otherwise hold
// registers across the loops).


// Shared pieces of the two passes. A score tile t[8] of a wave holds, for
// lane (lq = lane % 16, g = lane / 16), the 4 rows 16 j + 4 g + r (r = 0..3;
// rows: the 128-long side) of column lq of a 16-column block.
constexpr int BNT = 512;   // eight waves of 16 columns

template <int D>
struct BwdTile {
  static constexpr int KH = D / 64, KS = D / 32, DB = D / 16;
  using DK = Direct<true, FT, BNT>;            // one 64-dim half: [128 rows][64]
  static constexpr int IMG = KH * DK::BYTES;   // a [128 rows][D] K-major image
  static constexpr int SCL = D + 8;            // strip row (elements), padded
  static constexpr int STRIP = 16 * SCL * 2;   // 16 checksum rows of D
  static constexpr int RSTRIP = FT * 4 * 2;    // [128 rows][4] row-checksum strip
  static constexpr int ZERO = 64;              // zeros the strips' other 12 columns read
  static constexpr int SCR = 160;              // floats of rare-path scratch per wave
  static constexpr int NSV = 1024 / BNT;       // strip values staged per thread
  __host__ __device__ static constexpr int align1k(int x) { return (x + 1023) & ~1023; }

  // the fragment of two transposing reads through the compiler's
  // intrinsic (it tracks their completion itself: no wait is forced here)
  __device__ static __forceinline__ bf16x8 join(const TrPair& t) {
    typedef short short8_t __attribute__((ext_vector_type(8)));
    const short8_t v = {t.lo[0], t.lo[1], t.lo[2], t.lo[3], t.hi[0], t.hi[1], t.hi[2], t.hi[3]};
    return __builtin_bit_cast(bf16x8, v);
  }
  // transposed operand fragment (rows: dims rb + lane % 16; k: image rows
  // kb + 4g + 0..3 and kb + 16 + 4g + 0..3) from a K-major image
  __device__ static __forceinline__ bf16x8 t_frag(const char* img, int rb, int kb, int lane) {
    const int s = lane & 15, g = lane >> 4;
    const int k1 = kb + 4 * g + (s >> 2), k2 = k1 + 16;
    const int m = rb + 4 * (s & 3);
    const char* half = img + (m >> 6) * DK::BYTES;
    const int mm = m & 63, c = mm >> 3, off = (mm & 7) * 2;
    return join(tr_pair_intrinsic(half + k1 * 128 + ((c ^ (k1 & 7)) << 4) + off,
                                  half + k2 * 128 + ((c ^ (k2 & 7)) << 4) + off));
  }
  // the same from a [128 rows][4] row-checksum strip as the 16-row operand
  // (rows 4..15 read zeros)
  __device__ static __forceinline__ bf16x8 rs_frag(const bf16_t* rs, const bf16_t* zeros, int kb,
                                                   int lane) {
    const int s = lane & 15, g = lane >> 4;
    const int k1 = kb + 4 * g + (s >> 2), k2 = k1 + 16;
    const bool real = (s & 3) == 0;
    return join(tr_pair_intrinsic(real ? rs + k1 * 4 : zeros, real ? rs + k2 * 4 : zeros));
  }
  // the operand of the packed 32-row slab t of a packed tile
  __device__ static __forceinline__ bf16x8 slab(const uint2 (&pk)[8], int t) {
    const uint4 u = {pk[2 * t].x, pk[2 * t].y, pk[2 * t + 1].x, pk[2 * t + 1].y};
    return __builtin_bit_cast(bf16x8, u);
  }
  __device__ static __forceinline__ uint2 pack4(const float (&a)[4]) {
    return uint2{pack2(a[0], a[1]), pack2(a[2], a[3])};
  }
  __device__ static __forceinline__ uint2 pack4v(const float (&a)[4]) {
    return uint2{pack2v(a[0], a[1]), pack2v(a[2], a[3])};
  }
  __device__ static __forceinline__ void unpack4(uint2 p, float (&a)[4]) {
    a[0] = __uint_as_float(p.x << 16);
    a[1] = __uint_as_float(p.x & 0xffff0000u);
    a[2] = __uint_as_float(p.y << 16);
    a[3] = __uint_as_float(p.y & 0xffff0000u);
  }

  // Check of a score tile per (column, R-row block) against the strip
  // result cs (rows 4b..4b+3 of lane group b: hi/lo of c1, c2); columns are
  // entities cbase + 0..15, rows rbase + 0..127 (see score_locate for A, Bm
  // and tr). A flagged vector is gathered into the wave's scratch and fixed
  // by lane 0; the fixed element is put back into the tile.
  template <bool TR>
  __device__ static void check(floatx4 (&t)[8], const floatx4& cs, const FusedBwdDesc& fd, int op,
                               int b, int h, int cbase, int rbase, const bf16_t* A,
                               const bf16_t* Bm, int64_t lda, int64_t ldb, float* scr, int lane) {
    const int lq = lane & 15, g = lane >> 4;
    const int R = fd.R, NB = FT / R, lg_jpb = __builtin_ctz(R / 16);
    float mine1 = 0.f, minea = 0.f;
    if constexpr (D == 64) {
      // Each column's sums over the rows of every R-row block on the matrix
      // cores: the values and their magnitudes packed to bf16 (a rounding of
      // 2^-9 relative, far inside the detection bound E) as the B operand,
      // one slab of 32 rows per MFMA, against a block-indicator A operand
      // whose row 4 b is block b's: row 4 b of the result, register 0 of
      // lane group b, is block b's sum.
      floatx4 vs = {0.f, 0.f, 0.f, 0.f}, as = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float a0[4], a1[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) { a0[r] = t[2 * q][r]; a1[r] = t[2 * q + 1][r]; }
        const uint2 p0 = pack4v(a0), p1 = pack4v(a1);
        const uint4 u = {p0.x, p0.y, p1.x, p1.y};
        const uint4 ua = {u.x & 0x7fff7fffu, u.y & 0x7fff7fffu, u.z & 0x7fff7fffu, u.w & 0x7fff7fffu};
        const uint32_t one = lq == 4 * ((32 * q) >> (lg_jpb + 4)) ? 0x3f803f80u : 0u;
        const bf16x8 ind = __builtin_bit_cast(bf16x8, uint4{one, one, one, one});
        vs = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ind, __builtin_bit_cast(bf16x8, u), vs, 0, 0, 0);
        as = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ind, __builtin_bit_cast(bf16x8, ua), as, 0, 0, 0);
      }
      mine1 = vs[0];
      minea = as[0];
    } else {
      // the same sums on the vector ALUs (head dim 128: the matrix-core
      // form holds registers the key pass does not have)
      float sj[8], aj[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        sj[j] = (t[j][0] + t[j][1]) + (t[j][2] + t[j][3]);
        aj[j] = (fabsf(t[j][0]) + fabsf(t[j][1])) + (fabsf(t[j][2]) + fabsf(t[j][3]));
      }
      float r1[4], ra[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        r1[i] = sj[2 * i] + sj[2 * i + 1];
        ra[i] = aj[2 * i] + aj[2 * i + 1];
      }
      if (lg_jpb >= 2) {
        r1[0] += r1[1]; ra[0] += ra[1];
        r1[1] = r1[2] + r1[3]; ra[1] = ra[2] + ra[3];
      }
      if (lg_jpb >= 3) { r1[0] += r1[1]; ra[0] += ra[1]; }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (i < NB) {
          const float t1 = group4_sum(r1[i]), ta = group4_sum(ra[i]);
          if (g == i) { mine1 = t1; minea = ta; }
        }
      }
    }
    const float c1 = cs[0] + cs[1];
    uint64_t mask = __ballot(g < NB && flagged(c1 - mine1, minea, fd.e_rel));
    if (mask) {  // rare
      // the tile waits in private memory (indexed at run time, so it stays
      // there): none of its registers is live while the flagged vectors are
      // corrected
      float tm[8][4];
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) tm[j][r] = t[j][r];
      const float cs1 = cs[0] + cs[1], cs2 = cs[2] + cs[3];
      const int jpb = 1 << lg_jpb;
      while (mask) {
        const int L = __builtin_ctzll(mask);
        mask &= mask - 1;
        const int vq = L & 15, vb = L >> 4;
        if (lq == vq) {
          for (int jj = 0; jj < jpb; ++jj) {
            const int j = vb * jpb + jj;
#pragma unroll
            for (int r = 0; r < 4; ++r) scr[16 * jj + 4 * g + r] = tm[j][r];
          }
        }
        const float v1 = __shfl(cs1, L, 64);
        const float v2 = __shfl(cs2, L, 64);
        wave_sync_lds();
        score_locate(scr, R, v1, v2, fd.e_rel, fd.tn_s, fd.tc, fd.recompute, fd.report, op, b,
                     h, cbase + vq, rbase + vb * R, TR, lane);
        wave_sync_lds();
        if (fd.recompute && __float_as_int(scr[R]) >= 0) {
          const float nv = score_dot(A, Bm, lda, ldb, cbase + vq, rbase + vb * R +
                                     __float_as_int(scr[R]), D, lane);
          score_close(scr, R, nv, v1, fd.e_rel, fd.tn_s, fd.report, op, b, h, cbase + vq,
                      rbase + vb * R, TR, lane);
          wave_sync_lds();
        }
        const int idx = __float_as_int(scr[R]);
        const float nv = scr[R + 1];
        if (idx >= 0) {
          const int kl = vb * R + idx;
          if (lane == vq + 16 * ((kl & 15) >> 2)) tm[kl >> 4][kl & 3] = nv;
        }
        wave_sync_lds();
      }
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) t[j][r] = tm[j][r];
    }
  }

  // injected faults of op (test-only) on a score tile (coordinates as in
  // check: fault rows are queries and columns keys)
  template <bool TR>
  __device__ static void inject(floatx4 (&t)[8], const FusedBwdDesc& fd, int op, int b, int h,
                                int cbase, int rbase, int lane) {
    for (int f = 0; f < fd.n_faults; ++f) {
      const abft_fault ft = fd.faults[f];
      if (ft.op != op || ft.b != b || ft.h != h) continue;
      // under the mask only the block-lower-triangular region is computed
      if (fd.causal && ft.col / fd.R > ft.row / fd.R) continue;
      const int ci = (TR ? ft.col : ft.row) - cbase, ri = (TR ? ft.row : ft.col) - rbase;
      if (ci < 0 || ci >= 16 || ri < 0 || ri >= FT) continue;
      const int olane = ci + 16 * ((ri & 15) >> 2);
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (lane == olane && j == (ri >> 4) && r == (ri & 3))
            t[j][r] = ft.mode == ABFT_FAULT_FLIP ? flip_f32(t[j][r]) : ft.value;
    }
  }

  // A gradient's transposed accumulators acc[DB] (lane: dims 16 db + 4 g + r
  // of entity cbase + lq) and its strip result chk (lane group 0: hi/lo of
  // the sum and of the 1-based weighted sum over the dims): rounded, faults
  // of op injected, each entity's row checked (a located element fixed
  // from the checksum, Sec. 4.2) and stored at out + entity * ld.
  __device__ static void finish(floatx4 (&acc)[DB], const floatx4& chk, const FusedBwdDesc& fd,
                                bool check, bool wf, int op, int b, int h, int cbase, bf16_t* out,
                                int64_t ld, float* scr, int lane) {
    const int lq = lane & 15, g = lane >> 4;
    {
      const int e = cbase + lq;
      float ov[DB][4];
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 4; ++r) ov[db][r] = bf2f(f2bf(acc[db][r]));
      if (wf) {
        for (int f = 0; f < fd.n_faults; ++f) {
          const abft_fault ft = fd.faults[f];
          if (ft.op != op || ft.b != b || ft.h != h || ft.row != e) continue;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (ft.col == 16 * db + 4 * g + r)
                ov[db][r] = ft.mode == ABFT_FAULT_FLIP ? bf2f(flip_exponent_msb(f2bf(ov[db][r])))
                                                       : bf2f(f2bf(ft.value));
        }
      }
      if (check) {
        const float c1 = __shfl(chk[0] + chk[1], lq, 64);
        const float c2 = __shfl(chk[2] + chk[3], lq, 64);
        float r1 = 0.f, ra = 0.f;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            r1 += ov[db][r];
            ra += fabsf(ov[db][r]);
          }
        r1 = group4_sum(r1);
        ra = group4_sum(ra);
        uint64_t mask = __ballot(g == 0 && flagged(c1 - r1, ra, fd.e_rel));
        while (mask) {
          const int L = __builtin_ctzll(mask);
          mask &= mask - 1;
          if (lq == L) {
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
              for (int r = 0; r < 4; ++r) scr[16 * db + 4 * g + r] = ov[db][r];
          }
          const float v1 = __shfl(c1, L, 64), v2 = __shfl(c2, L, 64);
          wave_sync_lds();
          grad_fix(scr, D, v1, v2, fd.e_rel, fd.tn, fd.tc, fd.report, op, b, h, cbase + L, lane);
          wave_sync_lds();
          const int idx = __float_as_int(scr[D]);
          const float nv = scr[D + 1];
          if (idx >= 0 && lq == L) {
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (idx == 16 * db + 4 * g + r) ov[db][r] = nv;
          }
          wave_sync_lds();
        }
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const uint2 w = {pack2(ov[db][0], ov[db][1]), pack2(ov[db][2], ov[db][3])};
        *reinterpret_cast<uint2*>(out + int64_t(e) * ld + 16 * db + 4 * g) = w;
      }
    }
  }

  // checksum strip of 16 rows (4 per R-row block: hi/lo of the sum and of
  // the weighted sum) from fp32 column checksums; thread tid stages up to
  // NSV values in v[] (issue) and writes them (commit)
  __device__ static __forceinline__ void strip_issue(const float* cc, int64_t ldc, int64_t blk0,
                                                     int NB, int tid, float (&v)[NSV]) {
#pragma unroll
    for (int p = 0; p < NSV; ++p) {
      const int e = tid + p * BNT;
      const int ee = e < NB * 2 * D ? e : 0;
      const int blk = ee / (2 * D), c = (ee / D) & 1, dd = ee % D;
      v[p] = cc[((blk0 + blk) * 2 + c) * ldc + dd];
    }
  }
  __device__ static __forceinline__ void strip_commit(bf16_t* st, int NB, int tid,
                                                      const float (&v)[NSV]) {
#pragma unroll
    for (int p = 0; p < NSV; ++p) {
      const int e = tid + p * BNT;
      if (e < NB * 2 * D) {
        const int blk = e / (2 * D), c = (e / D) & 1, dd = e % D;
        const int r = (4 * blk + 2 * c) * SCL + dd;
        st[r] = f2bf(v[p]);
        st[r + SCL] = f2bf(v[p] - bf2f(f2bf(v[p])));
      }
    }
  }
  // Row checksums over the head dims (the sum and the 1-based weighted
  // sum) of the 128 rows row0.. of a row-major [rows][ld] bf16 tensor, as
  // the hi/lo bf16 pairs of a [128 rows][4] strip: four threads per row,
  // D / 4 dims each, loaded with the tile (rstrip_issue) and summed when
  // it has landed (rstrip_commit).
  static constexpr int CPP = D / 32;  // 8-element chunks per thread
  __device__ static __forceinline__ void rstrip_issue(const bf16_t* base, int64_t ld, int row0,
                                                      int nrows, int tid, bf16x8 (&v)[CPP]) {
    const bf16_t* p = base + int64_t(min(row0 + (tid >> 2), nrows - 1)) * ld + (tid & 3) * (8 * CPP);
#pragma unroll
    for (int cc = 0; cc < CPP; ++cc) v[cc] = *reinterpret_cast<const bf16x8*>(p + 8 * cc);
  }
  __device__ static __forceinline__ void rstrip_commit(bf16_t* rs, int tid, const bf16x8 (&v)[CPP]) {
    const int row = tid >> 2, part = tid & 3;
    // two elements per step: dot products of bf16 pairs with (1, 1) and
    // with their 1-based indices in the thread's range
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 ones = {__bf16(1.f), __bf16(1.f)};
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int cc = 0; cc < CPP; ++cc) {
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const bf16x2 x = {v[cc][e], v[cc][e + 1]};
        const bf16x2 w = {__bf16(float(8 * cc + e + 1)), __bf16(float(8 * cc + e + 2))};
        s1 = __builtin_amdgcn_fdot2_f32_bf16(x, ones, s1, false);
        s2 = __builtin_amdgcn_fdot2_f32_bf16(x, w, s2, false);
      }
    }
    s2 = fmaf(float(8 * CPP * part), s1, s2);    // the range starts at dim 8 CPP part
    s1 += __shfl_xor(s1, 1, 64);
    s2 += __shfl_xor(s2, 1, 64);
    s1 += __shfl_xor(s1, 2, 64);
    s2 += __shfl_xor(s2, 2, 64);
    if (part == 0) {
      const uint2 w = {pack2(s1, s1 - bf2f(f2bf(s1))), pack2(s2, s2 - bf2f(f2bf(s2)))};
      *reinterpret_cast<uint2*>(rs + row * 4) = w;
    }
  }
};

// The query pass. LDS: per key tile a stage of the K and V images and the
// K^c, V^c and K^r strips (two stages at head dim 64: the next tile loads
// while this one is used), the workgroup's Q and dCL images (loaded once),
// scratch.
template <int D, bool CHK>
struct FusedBwdQ : BwdTile<D> {
  using T = BwdTile<D>;
  using typename T::DK;
  static constexpr int KS = T::KS, DB = T::DB, KH = T::KH, IMG = T::IMG, SCL = T::SCL;
  static constexpr int NBUF = D == 64 ? 2 : 1;
  // offsets within a stage
  static constexpr int OFF_V = IMG, OFF_KC = 2 * IMG, OFF_VC = OFF_KC + T::STRIP;
  static constexpr int OFF_KR = OFF_VC + T::STRIP;
  static constexpr int STAGE = T::align1k(OFF_KR + T::RSTRIP);
  static constexpr int OFF_ZERO = NBUF * STAGE;
  static constexpr int OFF_Q = T::align1k(OFF_ZERO + T::ZERO), OFF_G = OFF_Q + IMG;
  static constexpr int OFF_SCR = OFF_G + IMG;
  static constexpr int LDS_BYTES = OFF_SCR + (BNT / 64) * T::SCR * 4;
  static_assert(LDS_BYTES <= 160 * 1024, "one workgroup fits the LDS");

  __device__ static void run(const FusedBwdDesc& fd, char* smem) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lq = lane & 15, g = lane >> 4;
    const int S = fd.S, H = fd.H, R = fd.R, NB = FT / R, nqR = S / R;
    const int nqt = S / FT, nbh = fd.B * fd.nh;
    const int z = blockIdx.x % nbh;
    const int qt = fd.causal ? nqt - 1 - int(blockIdx.x) / nbh : int(blockIdx.x) / nbh;
    const int b = z / fd.nh, h = z % fd.nh;
    const int q0 = qt * FT, qw = q0 + wave * 16, q = qw + lq;
    const int64_t ld = 3 * int64_t(H);
    const bf16_t* base = static_cast<const bf16_t*>(fd.qkv) + int64_t(b) * S * ld;
    const bf16_t* Qp = base + h * D;
    const bf16_t* Kp = base + H + h * D;
    const bf16_t* Vp = base + 2 * H + h * D;
    const bf16_t* dCLp = static_cast<const bf16_t*>(fd.dcl) + int64_t(b) * S * H + h * D;
    const bf16_t* CLp = static_cast<const bf16_t*>(fd.cl) + int64_t(b) * S * H + h * D;
    const int nkt = fd.causal ? qt + 1 : nqt;
    const float sl2 = fd.scale * 1.4426950408889634f;
    constexpr bool chk = CHK;
    const bool wf = fd.n_faults > 0 &&
                    faults_at(fd.faults, fd.n_faults, b, h,
                              (1u << ABFT_OP_AS) | (1u << ABFT_OP_DAP) | (1u << ABFT_OP_DQ));

    // the statistics and the softmax backward's row term D = dCL . CL of
    // the lane's query (D also kept for the key pass)
    float mq, il, ml, dq, sdq;
    {
      float acc = 0.f;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const bf16x8 gv = *reinterpret_cast<const bf16x8*>(dCLp + int64_t(q) * H + 32 * kk + 8 * g);
        const bf16x8 cv = *reinterpret_cast<const bf16x8*>(CLp + int64_t(q) * H + 32 * kk + 8 * g);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = fmaf(float(gv[e]), float(cv[e]), acc);
      }
      dq = group4_sum(acc);
      const float* st = fd.stats + ((int64_t(b) * fd.nh + h) * S + q) * 2;
      mq = st[0];
      il = 1.f / st[1];
      ml = mq + __log2f(st[1]);  // P = exp2(scaled score - ml)
      sdq = fd.scale * dq;       // dS = P (scale dP - scale D)
      if (g == 0) fd.drow[(int64_t(b) * fd.nh + h) * S + q] = dq;
    }
    // Q and dCL images of the workgroup's queries (complete with tile 0)
#pragma unroll
    for (int hf = 0; hf < KH; ++hf) {
      DK::issue(Qp, ld, q0, S, hf * 64, smem + OFF_Q + hf * DK::BYTES, wave, lane);
      DK::issue(dCLp, H, q0, S, hf * 64, smem + OFF_G + hf * DK::BYTES, wave, lane);
    }
    const bf16_t* zeros = reinterpret_cast<const bf16_t*>(smem + OFF_ZERO);
    if (chk && tid < T::ZERO / 4) reinterpret_cast<uint32_t*>(smem + OFF_ZERO)[tid] = 0u;

    // loads of key tile kt into stage st: the images by direct-to-LDS
    // copies, the strips' values into registers (written by commit)
    float kcv[T::NSV], vcv[T::NSV];
    bf16x8 krv[T::CPP];
    auto issue = [&](int kt, int st) {
      const int key0 = kt * FT;
      if (chk) {
        const int64_t blk0 = int64_t(b) * nqR + key0 / R;
        T::strip_issue(fd.qkvc + H + h * D, ld, blk0, NB, tid, kcv);
        T::strip_issue(fd.qkvc + 2 * H + h * D, ld, blk0, NB, tid, vcv);
        T::rstrip_issue(Kp, ld, key0, S, tid, krv);
      }
      char* sb = smem + st * STAGE;
#pragma unroll
      for (int hf = 0; hf < KH; ++hf) {
        DK::issue(Kp, ld, key0, S, hf * 64, sb + hf * DK::BYTES, wave, lane);
        DK::issue(Vp, ld, key0, S, hf * 64, sb + OFF_V + hf * DK::BYTES, wave, lane);
      }
    };
    auto commit = [&](int st) {
      if (chk) {
        char* sb = smem + st * STAGE;
        T::strip_commit(reinterpret_cast<bf16_t*>(sb + OFF_KC), NB, tid, kcv);
        T::strip_commit(reinterpret_cast<bf16_t*>(sb + OFF_VC), NB, tid, vcv);
        T::rstrip_commit(reinterpret_cast<bf16_t*>(sb + OFF_KR), tid, krv);
      }
    };

    floatx4 dqa[DB], kra = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int db = 0; db < DB; ++db) dqa[db] = floatx4{0.f, 0.f, 0.f, 0.f};
    float* scr = reinterpret_cast<float*>(smem + OFF_SCR) + wave * T::SCR;
    // B operand fragment of the wave's queries (rows of the Q or dCL image)
    auto bfrag = [&](int off, int kk) {
      return DK::frag(smem + off + (kk >> 1) * DK::BYTES, wave * 16, (kk & 1) * 32, lane);
    };

    if (NBUF == 2) {
      issue(0, 0);
      wait_vmcnt<0>();
      commit(0);
    }
    for (int kt = 0; kt < nkt; ++kt) {
      const int st = NBUF == 2 ? (kt & 1) : 0;
      if (NBUF == 1) {
        issue(kt, 0);
        wait_vmcnt<0>();
        commit(0);
      }
      // tile kt in LDS (double-buffered: the other stage is free)
      __syncthreads();
      const bool pre = NBUF == 2 && kt + 1 < nkt;
      if (pre) issue(kt + 1, st ^ 1);
      const char* sb = smem + st * STAGE;
      const bf16_t* krs = reinterpret_cast<const bf16_t*>(sb + OFF_KR);
      const int key0 = kt * FT;
      const bool diag = fd.causal && kt == qt;
      // P^T, then dS^T, packed to bf16: pk[j] holds keys 16 j + 4 g + 0..3
      uint2 pk[8];
      {
        // S^T = K Q^T with its strip rows, checked; P from the statistics
        floatx4 s[8], ks = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 8; ++j) s[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          const bf16x8 qf = bfrag(OFF_Q, kk);
          const char* sk = sb + (kk >> 1) * DK::BYTES;
#pragma unroll
          for (int j = 0; j < 8; ++j)
            s[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(DK::frag(sk, 16 * j, (kk & 1) * 32, lane),
                                                           qf, s[j], 0, 0, 0);
          if (chk) {
            const bf16_t* kcs = reinterpret_cast<const bf16_t*>(sb + OFF_KC);
            ks = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                *reinterpret_cast<const bf16x8*>(kcs + lq * SCL + 32 * kk + 8 * g), qf, ks, 0, 0, 0);
          }
        }
        if (wf) T::template inject<false>(s, fd, ABFT_OP_AS, b, h, qw, key0, lane);
        if (chk)
          T::template check<false>(s, ks, fd, ABFT_OP_AS, b, h, qw, key0, Qp, Kp, ld, ld, scr, lane);
        // masked keys (diagonal tile only) enter the exponential as -inf
        auto probs = [&](auto masked) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            float a[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool cut = masked && key0 + 16 * j + 4 * g + r > q;
              a[r] = __builtin_amdgcn_exp2f(cut ? -INFINITY : s[j][r] * sl2 - ml);
            }
            pk[j] = T::pack4v(a);
          }
        };
        // (head dim 64: a copy without the mask for the other tiles; head
        // dim 128: one copy, per element, as its registers allow)
        if constexpr (D == 64) {
          if (diag)
            probs(std::true_type{});
          else
            probs(std::false_type{});
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            float a[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool live = !(diag && key0 + 16 * j + 4 * g + r > q);
              a[r] = live ? bf2f(f2bf(__builtin_amdgcn_exp2f(s[j][r] * sl2 - mq) * il)) : 0.f;
            }
            pk[j] = T::pack4(a);
          }
        }
      }
      {
        // dP^T = V dCL^T with its strip rows, checked; dS from P and dP
        floatx4 dp[8], vs = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 8; ++j) dp[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          const bf16x8 gf = bfrag(OFF_G, kk);
          const char* sv = sb + OFF_V + (kk >> 1) * DK::BYTES;
#pragma unroll
          for (int j = 0; j < 8; ++j)
            dp[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(DK::frag(sv, 16 * j, (kk & 1) * 32, lane),
                                                            gf, dp[j], 0, 0, 0);
          if (chk) {
            const bf16_t* vcs = reinterpret_cast<const bf16_t*>(sb + OFF_VC);
            vs = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                *reinterpret_cast<const bf16x8*>(vcs + lq * SCL + 32 * kk + 8 * g), gf, vs, 0, 0, 0);
          }
        }
        if (wf) T::template inject<false>(dp, fd, ABFT_OP_DAP, b, h, qw, key0, lane);
        if (chk)
          T::template check<false>(dp, vs, fd, ABFT_OP_DAP, b, h, qw, key0, dCLp, Vp, H, ld, scr,
                                   lane);
        auto grads = [&](auto masked) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            float a[4], ds[4];
            T::unpack4(pk[j], a);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool cut = masked && key0 + 16 * j + 4 * g + r > q;
              ds[r] = cut ? 0.f : a[r] * fmaf(fd.scale, dp[j][r], -sdq);
            }
            pk[j] = T::pack4v(ds);
          }
        };
        // (head dim 64: a copy without the mask for the other tiles; head
        // dim 128: one copy, per element, as its registers allow)
        if constexpr (D == 64) {
          if (diag)
            grads(std::true_type{});
          else
            grads(std::false_type{});
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            float a[4], ds[4];
            T::unpack4(pk[j], a);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool live = !(diag && key0 + 16 * j + 4 * g + r > q);
              ds[r] = live ? bf2f(f2bf(fd.scale * a[r] * (dp[j][r] - dq))) : 0.f;
            }
            pk[j] = T::pack4(ds);
          }
        }
      }
      // the next tile's strips into the free stage
      if (pre) commit(st ^ 1);
      // dQ^T += K^T dS^T and (dQ^r)^T += (K^r)^T dS^T
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const bf16x8 pf = T::slab(pk, t);
#pragma unroll
        for (int db = 0; db < DB; ++db)
          dqa[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(T::t_frag(sb, 16 * db, 32 * t, lane),
                                                            pf, dqa[db], 0, 0, 0);
        if (chk)
          kra = __builtin_amdgcn_mfma_f32_16x16x32_bf16(T::rs_frag(krs, zeros, 32 * t, lane), pf,
                                                        kra, 0, 0, 0);
      }
      if (NBUF == 2)
        wait_vmcnt<0>();  // the next tile's copies
      else
        __syncthreads();  // the one stage is reloaded next
    }

    bf16_t* dQp = static_cast<bf16_t*>(fd.dqkv) + int64_t(b) * S * fd.ld + h * D;
    T::finish(dqa, kra, fd, chk, wf, ABFT_OP_DQ, b, h, qw, dQp, fd.ld, scr, lane);
  }
};

// The key pass. LDS: the workgroup's K and V images (loaded once); per
// query tile a stage of the Q and dCL images, the Q^c and dCL^c strips,
// the Q^r and dCL^r row-checksum strips and the queries' max, 1 / sum and D
// (two stages at head dim 64: the next tile loads while this one is used);
// scratch.
// PART 0 forms dV and dK together; where both sets of accumulators do not
// fit the registers of two waves per SIMD (head dim 128) the pass runs as
// PART 1 (S, P, dV) then PART 2 (S, P, dP, dS, dK), each recomputing and
// checking the scores; injected score faults are applied in the part that
// also forms dP, so that a fault is met once per pass whatever the split.
template <int D, bool CHK, int PART>
struct FusedBwdKV : BwdTile<D> {
  using T = BwdTile<D>;
  using typename T::DK;
  static constexpr int KS = T::KS, DB = T::DB, KH = T::KH, IMG = T::IMG, SCL = T::SCL;
  static constexpr int NBUF = D == 64 ? 2 : 1;
  static constexpr int OFF_V = IMG, OFF_ST = 2 * IMG;
  // offsets within a stage
  static constexpr int OFF_Q = 0, OFF_G = IMG;
  static constexpr int OFF_QC = 2 * IMG, OFF_GC = OFF_QC + T::STRIP;
  static constexpr int OFF_QR = OFF_GC + T::STRIP, OFF_GR = OFF_QR + T::RSTRIP;
  static constexpr int OFF_ROW = OFF_GR + T::RSTRIP;            // [3][128] floats
  static constexpr int STAGE = T::align1k(OFF_ROW + 3 * FT * 4);
  static constexpr int OFF_ZERO = OFF_ST + NBUF * STAGE;
  static constexpr int OFF_SCR = OFF_ZERO + T::ZERO;
  static constexpr int LDS_BYTES = OFF_SCR + (BNT / 64) * T::SCR * 4;
  static_assert(LDS_BYTES <= 160 * 1024, "one workgroup fits the LDS");

  __device__ static void run(const FusedBwdDesc& fd, char* smem) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lq = lane & 15, g = lane >> 4;
    const int S = fd.S, H = fd.H, R = fd.R, NB = FT / R, nqR = S / R;
    const int nqt = S / FT, nbh = fd.B * fd.nh;
    const int z = blockIdx.x % nbh;
    const int kt = int(blockIdx.x) / nbh;   // causal: the first key tiles see the most queries
    const int b = z / fd.nh, h = z % fd.nh;
    const int key0 = kt * FT, kw = key0 + wave * 16, key = kw + lq;
    const int64_t ld = 3 * int64_t(H);
    const bf16_t* base = static_cast<const bf16_t*>(fd.qkv) + int64_t(b) * S * ld;
    const bf16_t* Qp = base + h * D;
    const bf16_t* Kp = base + H + h * D;
    const bf16_t* Vp = base + 2 * H + h * D;
    const bf16_t* dCLp = static_cast<const bf16_t*>(fd.dcl) + int64_t(b) * S * H + h * D;
    const int qt0 = fd.causal ? kt : 0;
    const float sl2 = fd.scale * 1.4426950408889634f;
    constexpr bool chk = CHK;
    const int64_t bh = int64_t(b) * fd.nh + h;
    constexpr bool DO_V = PART != 2, DO_K = PART != 1;
    const bool wf = fd.n_faults > 0 &&
                    faults_at(fd.faults, fd.n_faults, b, h,
                              (1u << ABFT_OP_AS) | (1u << ABFT_OP_DAP) | (1u << ABFT_OP_DK) |
                                  (1u << ABFT_OP_DV));

    // K and V images of the workgroup's keys (complete with the first tile)
#pragma unroll
    for (int hf = 0; hf < KH; ++hf) {
      DK::issue(Kp, ld, key0, S, hf * 64, smem + hf * DK::BYTES, wave, lane);
      DK::issue(Vp, ld, key0, S, hf * 64, smem + OFF_V + hf * DK::BYTES, wave, lane);
    }
    const bf16_t* zeros = reinterpret_cast<const bf16_t*>(smem + OFF_ZERO);
    if (chk && tid < T::ZERO / 4) reinterpret_cast<uint32_t*>(smem + OFF_ZERO)[tid] = 0u;

    float qcv[T::NSV], gcv[T::NSV];
    bf16x8 qrv[T::CPP], grv[T::CPP];
    float rv0 = 0.f, rv1 = 0.f;
    // loads of query tile qt into stage st: the images by direct-to-LDS
    // copies, the statistics' and strips' values into registers (written by
    // commit)
    auto issue_values = [&](int qt) {
      const int q0 = qt * FT;
      // threads 0..127: max and sum of query q0 + tid; 128..255: its D
      const int qi = q0 + (tid & (FT - 1));
      if (tid < FT) {
        rv0 = fd.stats[(bh * S + qi) * 2];
        rv1 = fd.stats[(bh * S + qi) * 2 + 1];
      } else if (tid < 2 * FT) {
        rv0 = fd.drow[bh * S + qi];
      }
      if (chk) {
        const int64_t blk0 = int64_t(b) * nqR + q0 / R;
        T::strip_issue(fd.qkvc + h * D, ld, blk0, NB, tid, qcv);
        T::strip_issue(fd.dclc + h * D, H, blk0, NB, tid, gcv);
        if (DO_K) T::rstrip_issue(Qp, ld, q0, S, tid, qrv);
        if (DO_V) T::rstrip_issue(dCLp, H, q0, S, tid, grv);
      }
    };
    auto issue_copies = [&](int qt, int st) {
      const int q0 = qt * FT;
      char* sb = smem + OFF_ST + st * STAGE;
#pragma unroll
      for (int hf = 0; hf < KH; ++hf) {
        DK::issue(Qp, ld, q0, S, hf * 64, sb + OFF_Q + hf * DK::BYTES, wave, lane);
        DK::issue(dCLp, H, q0, S, hf * 64, sb + OFF_G + hf * DK::BYTES, wave, lane);
      }
    };
    auto commit = [&](int st) {
      char* sb = smem + OFF_ST + st * STAGE;
      float* rowf = reinterpret_cast<float*>(sb + OFF_ROW);
      if (tid < FT) {
        // head dim 64: max + log2(sum), so that P = exp2(scaled score -
        // that); 128: the max and 1 / sum
        rowf[tid] = D == 64 ? rv0 + __log2f(rv1) : rv0;
        rowf[FT + tid] = 1.f / rv1;
      } else if (tid < 2 * FT) {
        // D per query (head dim 64: scale D, for dS = P (scale dP - scale D))
        rowf[2 * FT + tid - FT] = D == 64 ? fd.scale * rv0 : rv0;
      }
      if (chk) {
        T::strip_commit(reinterpret_cast<bf16_t*>(sb + OFF_QC), NB, tid, qcv);
        T::strip_commit(reinterpret_cast<bf16_t*>(sb + OFF_GC), NB, tid, gcv);
        if (DO_K) T::rstrip_commit(reinterpret_cast<bf16_t*>(sb + OFF_QR), tid, qrv);
        if (DO_V) T::rstrip_commit(reinterpret_cast<bf16_t*>(sb + OFF_GR), tid, grv);
      }
    };

    floatx4 dva[DB], dka[DB], vra = {0.f, 0.f, 0.f, 0.f}, kra = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      dva[db] = floatx4{0.f, 0.f, 0.f, 0.f};
      dka[db] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    float* scr = reinterpret_cast<float*>(smem + OFF_SCR) + wave * T::SCR;
    // A operand fragments of the tile's queries (rows 16 j..) and the B
    // operand fragment of the wave's keys (rows of the K or V image)
    auto afrag = [&](const char* img, int j, int kk) {
      return DK::frag(img + (kk >> 1) * DK::BYTES, 16 * j, (kk & 1) * 32, lane);
    };
    auto kfrag = [&](int off, int kk) {
      return DK::frag(smem + off + (kk >> 1) * DK::BYTES, wave * 16, (kk & 1) * 32, lane);
    };

    if (NBUF == 2) {
      issue_values(qt0);
      issue_copies(qt0, 0);
      wait_vmcnt<0>();
      commit(0);
    }
    for (int qt = qt0; qt < nqt; ++qt) {
      const int st = NBUF == 2 ? ((qt - qt0) & 1) : 0;
      if (NBUF == 1) {
        issue_values(qt);
        issue_copies(qt, 0);
        wait_vmcnt<0>();
        commit(0);
      }
      // query tile qt in LDS (double-buffered: the other stage is free)
      __syncthreads();
      const bool pre = NBUF == 2 && qt + 1 < nqt;
      if (pre) issue_copies(qt + 1, st ^ 1);
      const char* sb = smem + OFF_ST + st * STAGE;
      const float* rowf = reinterpret_cast<const float*>(sb + OFF_ROW);
      const bf16_t* qrs = reinterpret_cast<const bf16_t*>(sb + OFF_QR);
      const bf16_t* grs = reinterpret_cast<const bf16_t*>(sb + OFF_GR);
      const int q0 = qt * FT;
      const bool diag = fd.causal && qt == kt;
      // P, then dS, packed to bf16: pk[j] holds queries 16 j + 4 g + 0..3
      uint2 pk[8];
      {
        // S = Q K^T with its strip rows (Q^c) K^T, column-checked; P
        floatx4 s[8], cs = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 8; ++j) s[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          const bf16x8 kf = kfrag(0, kk);
#pragma unroll
          for (int j = 0; j < 8; ++j)
            s[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag(sb + OFF_Q, j, kk), kf, s[j], 0, 0, 0);
          if (chk) {
            const bf16_t* qcs = reinterpret_cast<const bf16_t*>(sb + OFF_QC);
            cs = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                *reinterpret_cast<const bf16x8*>(qcs + lq * SCL + 32 * kk + 8 * g), kf, cs, 0, 0, 0);
          }
        }
        if (DO_K && wf) T::template inject<true>(s, fd, ABFT_OP_AS, b, h, kw, q0, lane);
        if (chk)
          T::template check<true>(s, cs, fd, ABFT_OP_AS, b, h, kw, q0, Kp, Qp, ld, ld, scr, lane);
        // masked queries (diagonal tile only) enter the exponential as -inf
        auto probs = [&](auto masked) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float4 m4 = *reinterpret_cast<const float4*>(rowf + 16 * j + 4 * g);
            const float mv[4] = {m4.x, m4.y, m4.z, m4.w};
            float a[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool cut = masked && key > q0 + 16 * j + 4 * g + r;
              a[r] = __builtin_amdgcn_exp2f(cut ? -INFINITY : s[j][r] * sl2 - mv[r]);
            }
            pk[j] = T::pack4v(a);
          }
        };
        // (head dim 64: a copy without the mask for the other tiles; head
        // dim 128: one copy, per element, as its registers allow)
        if constexpr (D == 64) {
          if (diag)
            probs(std::true_type{});
          else
            probs(std::false_type{});
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float4 m4 = *reinterpret_cast<const float4*>(rowf + 16 * j + 4 * g);
            const float4 i4 = *reinterpret_cast<const float4*>(rowf + FT + 16 * j + 4 * g);
            const float mv[4] = {m4.x, m4.y, m4.z, m4.w}, iv[4] = {i4.x, i4.y, i4.z, i4.w};
            float a[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool live = !(diag && key > q0 + 16 * j + 4 * g + r);
              a[r] = live ? bf2f(f2bf(__builtin_amdgcn_exp2f(s[j][r] * sl2 - mv[r]) * iv[r])) : 0.f;
            }
            pk[j] = T::pack4(a);
          }
        }
      }
      // the next tile's values, written to the free stage at the end
      if (pre) issue_values(qt + 1);
      // dV^T += dCL^T P and (dV^r)^T += (dCL^r)^T P
#pragma unroll
      for (int t = 0; t < 4 && DO_V; ++t) {
        const bf16x8 pf = T::slab(pk, t);
#pragma unroll
        for (int db = 0; db < DB; ++db)
          dva[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              T::t_frag(sb + OFF_G, 16 * db, 32 * t, lane), pf, dva[db], 0, 0, 0);
        if (chk)
          vra = __builtin_amdgcn_mfma_f32_16x16x32_bf16(T::rs_frag(grs, zeros, 32 * t, lane), pf,
                                                        vra, 0, 0, 0);
      }
      if (DO_K) {
        // dP = dCL V^T with its strip rows (dCL^c) V^T, column-checked; dS
        floatx4 dp[8], cs = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 8; ++j) dp[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          const bf16x8 vf = kfrag(OFF_V, kk);
#pragma unroll
          for (int j = 0; j < 8; ++j)
            dp[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag(sb + OFF_G, j, kk), vf, dp[j], 0, 0, 0);
          if (chk) {
            const bf16_t* gcs = reinterpret_cast<const bf16_t*>(sb + OFF_GC);
            cs = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                *reinterpret_cast<const bf16x8*>(gcs + lq * SCL + 32 * kk + 8 * g), vf, cs, 0, 0, 0);
          }
        }
        if (wf) T::template inject<true>(dp, fd, ABFT_OP_DAP, b, h, kw, q0, lane);
        if (chk)
          T::template check<true>(dp, cs, fd, ABFT_OP_DAP, b, h, kw, q0, Vp, dCLp, ld, H, scr,
                                  lane);
        auto grads = [&](auto masked) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float4 d4 = *reinterpret_cast<const float4*>(rowf + 2 * FT + 16 * j + 4 * g);
            const float dv[4] = {d4.x, d4.y, d4.z, d4.w};
            float a[4], ds[4];
            T::unpack4(pk[j], a);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool cut = masked && key > q0 + 16 * j + 4 * g + r;
              ds[r] = cut ? 0.f : a[r] * fmaf(fd.scale, dp[j][r], -dv[r]);
            }
            pk[j] = T::pack4v(ds);
          }
        };
        // (head dim 64: a copy without the mask for the other tiles; head
        // dim 128: one copy, per element, as its registers allow)
        if constexpr (D == 64) {
          if (diag)
            grads(std::true_type{});
          else
            grads(std::false_type{});
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float4 d4 = *reinterpret_cast<const float4*>(rowf + 2 * FT + 16 * j + 4 * g);
            const float dv[4] = {d4.x, d4.y, d4.z, d4.w};
            float a[4], ds[4];
            T::unpack4(pk[j], a);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool live = !(diag && key > q0 + 16 * j + 4 * g + r);
              ds[r] = live ? bf2f(f2bf(fd.scale * a[r] * (dp[j][r] - dv[r]))) : 0.f;
            }
            pk[j] = T::pack4(ds);
          }
        }
      }
      // dK^T += Q^T dS and (dK^r)^T += (Q^r)^T dS
#pragma unroll
      for (int t = 0; t < 4 && DO_K; ++t) {
        const bf16x8 pf = T::slab(pk, t);
#pragma unroll
        for (int db = 0; db < DB; ++db)
          dka[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              T::t_frag(sb + OFF_Q, 16 * db, 32 * t, lane), pf, dka[db], 0, 0, 0);
        if (chk)
          kra = __builtin_amdgcn_mfma_f32_16x16x32_bf16(T::rs_frag(qrs, zeros, 32 * t, lane), pf,
                                                        kra, 0, 0, 0);
      }
      if (NBUF == 2) {
        if (pre) commit(st ^ 1);  // the next tile's values into the free stage
        wait_vmcnt<0>();          // and its copies
      } else {
        __syncthreads();  // the one stage is reloaded next
      }
    }

    bf16_t* outp = static_cast<bf16_t*>(fd.dqkv) + int64_t(b) * S * fd.ld + h * D;
    if (DO_K) T::finish(dka, kra, fd, chk, wf, ABFT_OP_DK, b, h, kw, outp + H, fd.ld, scr, lane);
    if (DO_V)
      T::finish(dva, vra, fd, chk, wf, ABFT_OP_DV, b, h, kw, outp + 2 * H, fd.ld, scr, lane);
  }
};

// eight waves, two per SIMD
template <int D, bool CHK>
__global__ __launch_bounds__(BNT) __attribute__((amdgpu_waves_per_eu(2)))
void fused_bwd_q_kernel(FusedBwdDesc fd) {
  extern __shared__ __align__(16) char smem[];
  FusedBwdQ<D, CHK>::run(fd, smem);
}

template <int D, bool CHK, int PART>
__global__ __launch_bounds__(BNT) __attribute__((amdgpu_waves_per_eu(2)))
void fused_bwd_kv_kernel(FusedBwdDesc fd) {
  extern __shared__ __align__(16) char smem[];
  FusedBwdKV<D, CHK, PART>::run(fd, smem);
}

template <int D, bool PROT>
__global__ __launch_bounds__((FusedAttn<D, PROT>::NTH)) __attribute__((amdgpu_waves_per_eu(2)))
void fused_attn_kernel(FusedDesc fd) {
  extern __shared__ __align__(16) char smem[];
  FusedAttn<D, PROT>::run(fd, smem);
}

template <int D, bool PROT>
hipError_t launch_d(const FusedDesc& fd, hipStream_t s) {
  using F = FusedAttn<D, PROT>;
  static bool attr = false;
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fused_attn_kernel<D, PROT>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             F::LDS_BYTES);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int64_t grid = int64_t(fd.B) * fd.nh * (fd.S / FT);
  if (grid == 0) return hipSuccess;
  auto kern = fused_attn_kernel<D, PROT>;
  hipLaunchKernelGGL(kern, dim3(unsigned(grid)), dim3(F::NTH), F::LDS_BYTES, s, fd);
  return hipGetLastError();
}

template <auto KERN>
hipError_t launch_bwd_kernel(const FusedBwdDesc& fd, int lds, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(KERN),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int64_t grid = int64_t(fd.B) * fd.nh * (fd.S / FT);
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(KERN, dim3(unsigned(grid)), dim3(BNT), lds, s, fd);
  return hipGetLastError();
}

}  // namespace

// shapes and operands both passes need
static bool bwd_desc_ok(const FusedBwdDesc& fd) {
  return fd.S % FT == 0 && fd.R >= 32 && FT % fd.R == 0 && fd.H == fd.nh * fd.D &&
         fd.qkv != nullptr && fd.dcl != nullptr && fd.stats != nullptr && fd.drow != nullptr &&
         fd.dqkv != nullptr && fd.ld >= 3 * int64_t(fd.H);
}

hipError_t launch_fused_bwd_q(const FusedBwdDesc& fd, hipStream_t s) {
  if (!bwd_desc_ok(fd) || fd.cl == nullptr || (fd.check && fd.qkvc == nullptr))
    return hipErrorInvalidValue;
  if (fd.D == 64)
    return fd.check ? launch_bwd_kernel<fused_bwd_q_kernel<64, true>>(fd, FusedBwdQ<64, true>::LDS_BYTES, s)
                    : launch_bwd_kernel<fused_bwd_q_kernel<64, false>>(fd, FusedBwdQ<64, false>::LDS_BYTES, s);
  if (fd.D == 128)
    return fd.check ? launch_bwd_kernel<fused_bwd_q_kernel<128, true>>(fd, FusedBwdQ<128, true>::LDS_BYTES, s)
                    : launch_bwd_kernel<fused_bwd_q_kernel<128, false>>(fd, FusedBwdQ<128, false>::LDS_BYTES, s);
  return hipErrorInvalidValue;
}

hipError_t launch_fused_bwd_kv(const FusedBwdDesc& fd, hipStream_t s) {
  if (!bwd_desc_ok(fd) ||
      (fd.check && (fd.qkvc == nullptr || fd.dclc == nullptr)))
    return hipErrorInvalidValue;
  if (fd.D == 64)
    return fd.check
               ? launch_bwd_kernel<fused_bwd_kv_kernel<64, true, 0>>(fd, FusedBwdKV<64, true, 0>::LDS_BYTES, s)
               : launch_bwd_kernel<fused_bwd_kv_kernel<64, false, 0>>(fd, FusedBwdKV<64, false, 0>::LDS_BYTES, s);
  if (fd.D == 128 && !fd.check)
    return launch_bwd_kernel<fused_bwd_kv_kernel<128, false, 0>>(fd, FusedBwdKV<128, false, 0>::LDS_BYTES, s);
  if (fd.D == 128) {
    hipError_t e = fd.check
        ? launch_bwd_kernel<fused_bwd_kv_kernel<128, true, 1>>(fd, FusedBwdKV<128, true, 1>::LDS_BYTES, s)
        : launch_bwd_kernel<fused_bwd_kv_kernel<128, false, 1>>(fd, FusedBwdKV<128, false, 1>::LDS_BYTES, s);
    if (e != hipSuccess) return e;
    return fd.check
        ? launch_bwd_kernel<fused_bwd_kv_kernel<128, true, 2>>(fd, FusedBwdKV<128, true, 2>::LDS_BYTES, s)
        : launch_bwd_kernel<fused_bwd_kv_kernel<128, false, 2>>(fd, FusedBwdKV<128, false, 2>::LDS_BYTES, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_fused_fwd(const FusedDesc& fd, hipStream_t s) {
  if (fd.S % FT != 0 || fd.R < 16 || FT % fd.R != 0 || fd.H != fd.nh * fd.D)
    return hipErrorInvalidValue;
  const bool prot = fd.check_as || fd.check_cl || fd.vr != nullptr;
  if (prot && fd.R < 32) return hipErrorInvalidValue;  // 4 strip rows per block, 16 rows
  if ((fd.check_as && fd.qkvc == nullptr) || (fd.check_cl && fd.vr == nullptr))
    return hipErrorInvalidValue;
  if (fd.D == 64) return prot ? launch_d<64, true>(fd, s) : launch_d<64, false>(fd, s);
  if (fd.D == 128) return prot ? launch_d<128, true>(fd, s) : launch_d<128, false>(fd, s);
  return hipErrorInvalidValue;
}

}  // namespace abft
