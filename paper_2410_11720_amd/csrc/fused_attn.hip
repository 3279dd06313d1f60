// Fused protected attention, forward: the score, softmax and context steps
// of the layer (Sec. 2.1 Eq. 1-2) with the S_AS and S_CL checks of
// Sec. 4.4, in an online-softmax form that keeps neither the scores AS nor
// the probabilities AP in memory (an extension: the paper stores both).
//
// One workgroup per (batch, head, tile of 128 queries); each of its four
// waves owns 32 queries. Key tiles of 128 keys pass through LDS in order
// (causal: up to the diagonal tile), double-buffered for head_dim 64. Per
// key tile each wave computes
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
// need a reduction across the 16 lanes of a query group per key; with the
// root check, Q errors (the 1R patterns only the column side locates) are
// corrected before this kernel, and 0D and 1C errors are located by the
// rows.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "abft_internal.hpp"
#include "abft_device.hpp"
#include "direct_lds.hpp"

namespace abft {
namespace {

constexpr int FT = 128;   // queries per workgroup, keys per key tile
constexpr int FNT = 256;  // four waves of 32 queries

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

template <int D, bool PROT>
struct FusedAttn {
  static constexpr int NSTAGE = D == 64 ? 2 : 1;
  static constexpr int KH = D / 64;    // 64-wide halves of the head dim (K images)
  static constexpr int KS = D / 32;    // k steps of the score product
  static constexpr int DB = D / 16;    // 16-row blocks of O^T
  using DK = Direct<true, FT>;         // K half [128 keys][64 dims], swizzled
  using DV = Direct<false, D>;         // V image [64 keys][D dims], swizzled
  static constexpr int K_BYTES = KH * DK::BYTES;
  static constexpr int V_BYTES = 2 * DV::BYTES;
  static constexpr int KCL = D + 8;    // K^c strip row (elements), padded
  static constexpr int KC_BYTES = PROT ? 16 * KCL * 2 : 0;
  static constexpr int VR_BYTES = PROT ? FT * 16 * 2 : 0;
  static constexpr int STAGE_BYTES = K_BYTES + V_BYTES + KC_BYTES + VR_BYTES;
  static constexpr int SCR = 160;      // floats of rare-path scratch per wave
  static constexpr int LDS_BYTES = NSTAGE * STAGE_BYTES + (PROT ? 4 * SCR * 4 : 0);
  static_assert(LDS_BYTES <= 80 * 1024, "two workgroups per CU");

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
    const int q0 = qt * FT, qw = q0 + wave * 32;
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

    // Q as the B operand of S^T: query qw + 16 qb + lane % 16, dims 32 kk + 8 g..
    bf16x8 qf[2][KS];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
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
            const int e = tid + p * FNT;
            const bool ok = e < NB * 2 * D;
            const int ee = ok ? e : 0;
            const int blk = ee / (2 * D), c = (ee / D) & 1, dd = ee % D;
            // (used by commit only where e is in range: no select here, which
            // would wait for the load, and with it for the tile's loads)
            kcv[p] = arg->qkvc[((int64_t(b) * nqR + key0 / R + blk) * 2 + c) * ld + H + h * D + dd];
          }
        }
        if (arg->vr != nullptr)
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
            const int e = tid + p * FNT;
            if (e < NB * 2 * D) {
              const int blk = e / (2 * D), c = (e / D) & 1, dd = e % D;
              const bf16_t hi = f2bf(kcv[p]);
              const bf16_t lo = f2bf(kcv[p] - bf2f(hi));
              kcs[(4 * blk + 2 * c) * KCL + dd] = hi;
              kcs[(4 * blk + 2 * c + 1) * KCL + dd] = lo;
            }
          }
        }
        if (arg->vr != nullptr) {
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
        for (int e = tid; e < FT * 12; e += FNT) vrs[(e / 12) * 16 + 4 + e % 12] = 0;
      }
    }

    floatx4 o[DB][2], vra[2];
    float m[2], l[2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
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
      floatx4 s[8][2], ks[2];
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) s[j][qb] = floatx4{0.f, 0.f, 0.f, 0.f};
      ks[0] = ks[1] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const char* sk = sb + (kk >> 1) * DK::BYTES;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const bf16x8 kf = DK::frag(sk, 16 * j, (kk & 1) * 32, lane);
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
            s[j][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[qb][kk], s[j][qb], 0, 0, 0);
        }
        if constexpr (PROT) {
          if (arg->check_as) {
            const bf16_t* kcs = reinterpret_cast<const bf16_t*>(sb + K_BYTES + V_BYTES);
            const bf16x8 sf = *reinterpret_cast<const bf16x8*>(kcs + lq * KCL + 32 * kk + 8 * g);
#pragma unroll
            for (int qb = 0; qb < 2; ++qb)
              ks[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sf, qf[qb][kk], ks[qb], 0, 0, 0);
          }
        }
      }

      // injected score faults (test-only), on the unrounded scores
      if (arg->n_faults > 0) {
        for (int f = 0; f < arg->n_faults; ++f) {
          const abft_fault ft = arg->faults[f];
          if (ft.op != ABFT_OP_AS || ft.b != b || ft.h != h) continue;
          const int qi = ft.row - qw, ki = ft.col - key0;
          if (qi < 0 || qi >= 32 || ki < 0 || ki >= FT) continue;
          const int oq = qi >> 4, olane = (qi & 15) + 16 * ((ki & 15) >> 2);
#pragma unroll
          for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int qb = 0; qb < 2; ++qb)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (lane == olane && qb == oq && j == (ki >> 4) && r == (ki & 3))
                  s[j][qb][r] = ft.mode == ABFT_FAULT_FLIP ? flip_f32(s[j][qb][r]) : ft.value;
        }
      }

      // row check of S per (query, R-key block)
      if constexpr (PROT) {
        if (arg->check_as) {
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            float sj[8], aj[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              sj[j] = (s[j][qb][0] + s[j][qb][1]) + (s[j][qb][2] + s[j][qb][3]);
              aj[j] = (fabsf(s[j][qb][0]) + fabsf(s[j][qb][1])) +
                      (fabsf(s[j][qb][2]) + fabsf(s[j][qb][3]));
            }
            // block sums (2, 4 or 8 groups of 16 keys), reduced over the 4 lanes
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
            float mine1 = 0.f, minea = 0.f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              if (i < NB) {
                const float t1 = group4_sum(r1[i]), ta = group4_sum(ra[i]);
                if (g == i) { mine1 = t1; minea = ta; }
              }
            }
            const float c1 = ks[qb][0] + ks[qb][1];
            const bool fl = g < NB && flagged(c1 - mine1, minea, arg->e_rel);
            uint64_t mask = __ballot(fl);
            while (mask) {  // rare: locate and correct inside the wave
              const int L = __builtin_ctzll(mask);
              mask &= mask - 1;
              const int vq = L & 15, vb = L >> 4;    // query lane, key block
              // gather the vector S[q][block vb] into the scratch
#pragma unroll
              for (int j = 0; j < 8; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  if (lq == vq && (j >> lg_jpb) == vb)
                    scr[(16 * j + 4 * g + r) - vb * R] = s[j][qb][r];
              const float v1 = __shfl(ks[qb][0] + ks[qb][1], L, 64);
              const float v2 = __shfl(ks[qb][2] + ks[qb][3], L, 64);
              wave_sync_lds();
              if (lane == 0) {
                const int q = qw + 16 * qb + vq;
                const EecResult res = eec_locate<float>(scr, 1, R, v1, v2, arg->e_rel, arg->tn_s);
                int idx = -1;
                float nv = 0.f;
                if (res.status == EEC_LOCATED) {
                  idx = res.index;
                  const int key = key0 + vb * R + idx;
                  const float old = scr[idx];
                  int action = ABFT_ACT_RECOMPUTE;
                  if (arg->recompute) {
                    float acc = 0.f;
                    for (int dd = 0; dd < D; ++dd)
                      acc = fmaf(bf2f(Qp[int64_t(q) * ld + dd]), bf2f(Kp[int64_t(key) * ld + dd]), acc);
                    nv = acc;
                  } else {
                    nv = fix_by_checksum<float>(scr, 1, R, idx, v1, res.d1, arg->tc, &action);
                  }
                  scr[idx] = nv;
                  record_event(arg->report, ABFT_OP_AS, b, h, q, key, classify(old, arg->tn_s), action,
                               old);
                }
                if (res.status != EEC_CLEAN && vec_flagged<float>(scr, 1, R, v1, arg->e_rel))
                  record_event(arg->report, ABFT_OP_AS, b, h, q, key0 + vb * R, ABFT_KIND_NONE,
                               ABFT_ACT_UNCORRECTABLE, 0.f);
                scr[R] = __int_as_float(idx);
                scr[R + 1] = nv;
              }
              wave_sync_lds();
              const int idx = __float_as_int(scr[R]);
              const float nv = scr[R + 1];
              if (idx >= 0) {
                const int kl = vb * R + idx;
#pragma unroll
                for (int j = 0; j < 8; ++j)
#pragma unroll
                  for (int r = 0; r < 4; ++r)
                    if (lane == vq + 16 * ((kl & 15) >> 2) && j == (kl >> 4) && r == (kl & 3))
                      s[j][qb][r] = nv;
              }
              wave_sync_lds();
            }
          }
        }
      }

      // online softmax, then O^T += V^T P^T (and the V^r rows)
      const bool diag = arg->causal && kt == qt;
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        const int q = qw + 16 * qb + lq;
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float x = s[j][qb][r] * sl2;
            if (diag && key0 + 16 * j + 4 * g + r > q) x = -INFINITY;
            s[j][qb][r] = x;
            mx = fmaxf(mx, x);
          }
        mx = xmax32(xmax16(mx));
        const float mn = fmaxf(m[qb], mx);
        const float alpha = __builtin_amdgcn_exp2f(m[qb] - mn);
        m[qb] = mn;
        float ls = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float p = __builtin_amdgcn_exp2f(s[j][qb][r] - mn);
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
        bf16x8 pf[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          const uint4 u = {pack2(s[2 * t][qb][0], s[2 * t][qb][1]),
                           pack2(s[2 * t][qb][2], s[2 * t][qb][3]),
                           pack2(s[2 * t + 1][qb][0], s[2 * t + 1][qb][1]),
                           pack2(s[2 * t + 1][qb][2], s[2 * t + 1][qb][3])};
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
          for (int qb = 0; qb < 2; ++qb)
            o[db][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[qb], o[db][qb], 0, 0, 0);
          cur = nxt;
        }
        if (with_vr && !(D == 64 && PROT)) cur = vr_frag(vrs, 32 * t, lane);
        if (with_vr) {
          lds_wait_all();
          const bf16x8 rf = tr_join(cur);
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
            vra[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rf, pf[qb], vra[qb], 0, 0, 0);
        }
      }
      if (NSTAGE == 1) __syncthreads();  // the one stage is reloaded next
    }

    // CL = O / l: round, check against A^r / l, store
    bf16_t* CLp = static_cast<bf16_t*>(arg->cl) + int64_t(b) * S * H + h * D;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
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
          cr[0] = (vra[qb][0] + vra[qb][1]) * inv;
          cr[1] = (vra[qb][2] + vra[qb][3]) * inv;
        }
      }
      float ov[DB][4];
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 4; ++r) ov[db][r] = bf2f(f2bf(o[db][qb][r] * inv));
      if (arg->n_faults > 0) {
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
            if (lane == 0) {
              const int qq = qw + 16 * qb + L;
              const EecResult res = eec_locate<float>(scr, 1, D, v1, v2, arg->e_rel, arg->tn_cl);
              int idx = -1;
              float nv = 0.f;
              if (res.status == EEC_LOCATED) {
                idx = res.index;
                const float old = scr[idx];
                int action = 0;
                nv = bf2f(f2bf(fix_by_checksum<float>(scr, 1, D, idx, v1, res.d1, arg->tc, &action)));
                scr[idx] = nv;
                record_event(arg->report, ABFT_OP_CL, b, h, qq, idx, classify(old, arg->tn_cl), action,
                             old);
              }
              if (res.status != EEC_CLEAN && vec_flagged<float>(scr, 1, D, v1, arg->e_rel))
                record_event(arg->report, ABFT_OP_CL, b, h, qq, 0, ABFT_KIND_NONE,
                             ABFT_ACT_UNCORRECTABLE, 0.f);
              scr[D] = __int_as_float(idx);
              scr[D + 1] = nv;
            }
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
    }
  }
};

// Fused backward core (after a fused forward, which keeps no scores). Per
// (batch, head, tile of 128 queries), each of the four waves owning 32
// queries, key tiles of 128 keys pass through LDS (K and V as K-major
// images, the K^c and V^c strips, and the strip of K^r, the row checksums
// of K over the head dims); per key tile each wave computes
//   S^T = K Q^T (AS^r = Q (K^c)^T from the strip) and checks every
//     (query, R-key block) vector, as the forward does;
//   P = exp2(log2(e) scale S - m) / l from the forward's statistics,
//     rounded, stored as AP with its row checksums AP^r;
//   dP^T = V dCL^T (dP^r = dCL (V^c)^T from the strip) and the same row
//     check;
//   dS = scale P (dP - D), D = dCL . CL per query, rounded, stored with
//     its row checksums dAS^r;
//   dQ^T += K^T dS^T and (dQ^r)^T += (K^r)^T dS^T, the K^T fragments read
//     from the K image with transposing reads in the key order of the
//     dS^T fragment a lane assembles from its accumulators.
// After the last key tile dQ is rounded, row-checked against dQ^r (a
// located element fixed from the checksum) and stored.
template <int D, bool CHK>
struct FusedBwd {
  static constexpr int KH = D / 64, KS = D / 32, DB = D / 16;
  using DK = Direct<true, FT>;                 // one 64-dim half: [128 keys][64]
  static constexpr int IMG = KH * DK::BYTES;   // a [128 keys][D] K-major image
  static constexpr int SCL = D + 8;            // strip row (elements), padded
  static constexpr int STRIP = 16 * SCL * 2;
  static constexpr int OFF_V = IMG, OFF_KC = 2 * IMG, OFF_VC = OFF_KC + STRIP;
  static constexpr int OFF_KR = OFF_VC + STRIP;
  static constexpr int STAGE_BYTES = OFF_KR + FT * 16 * 2;
  // the workgroup's Q and dCL rows, [128 queries][D] K-major images read as
  // the B operands of S^T and dP^T (loaded once)
  static constexpr int OFF_Q = STAGE_BYTES, OFF_G = OFF_Q + IMG;
  static constexpr int SCR = 160;              // floats of rare-path scratch per wave
  static constexpr int OFF_SCR = OFF_G + IMG;
  static constexpr int LDS_BYTES = OFF_SCR + 4 * SCR * 4;

  // K^T operand fragment (rows: dims rb + lane % 16; k: keys kb + 4g + 0..3
  // and kb + 16 + 4g + 0..3) from the K-major image
  __device__ static __forceinline__ TrPair kt_frag(const char* img, int rb, int kb, int lane) {
    const int s = lane & 15, g = lane >> 4;
    const int k1 = kb + 4 * g + (s >> 2), k2 = k1 + 16;
    const int m = rb + 4 * (s & 3);
    const char* half = img + (m >> 6) * DK::BYTES;
    const int mm = m & 63, c = mm >> 3, off = (mm & 7) * 2;
    return tr_pair_intrinsic(half + k1 * 128 + ((c ^ (k1 & 7)) << 4) + off,
                             half + k2 * 128 + ((c ^ (k2 & 7)) << 4) + off);
  }
  // (K^r)^T fragment from the [128 keys][16] strip, same key order
  __device__ static __forceinline__ TrPair kr_frag(const bf16_t* krs, int kb, int lane) {
    const int s = lane & 15, g = lane >> 4;
    const int k1 = kb + 4 * g + (s >> 2), k2 = k1 + 16;
    const int m = 4 * (s & 3);
    return tr_pair_intrinsic(krs + k1 * 16 + m, krs + k2 * 16 + m);
  }

  // Row check of a 128-key x 32-query tile t (keys along the lane's
  // registers) per (query, R-key block) against the strip result cs (rows
  // 4b..4b+3 of lane group b: hi/lo of c1, c2): a flagged vector is
  // gathered into the wave's scratch, located by EEC and its element
  // recomputed as the dot product of row q of A and row key of Bm (length
  // D, leading dimensions lda, ldb) or fixed from the checksums.
  __device__ static void check_tile(floatx4 (&t)[8][2], const floatx4 (&cs)[2],
                                    const FusedBwdDesc& fd, int op, int b, int h, int qw,
                                    int key0, const bf16_t* A, const bf16_t* Bm, int64_t lda,
                                    int64_t ldb, float* scr, int lane) {
    const int lq = lane & 15, g = lane >> 4;
    const int R = fd.R, NB = FT / R, lg_jpb = __builtin_ctz(R / 16);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      float sj[8], aj[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        sj[j] = (t[j][qb][0] + t[j][qb][1]) + (t[j][qb][2] + t[j][qb][3]);
        aj[j] = (fabsf(t[j][qb][0]) + fabsf(t[j][qb][1])) +
                (fabsf(t[j][qb][2]) + fabsf(t[j][qb][3]));
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
      float mine1 = 0.f, minea = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (i < NB) {
          const float t1 = group4_sum(r1[i]), ta = group4_sum(ra[i]);
          if (g == i) { mine1 = t1; minea = ta; }
        }
      }
      const float c1 = cs[qb][0] + cs[qb][1];
      const bool fl = g < NB && flagged(c1 - mine1, minea, fd.e_rel);
      uint64_t mask = __ballot(fl);
      while (mask) {  // rare: locate and correct inside the wave
        const int L = __builtin_ctzll(mask);
        mask &= mask - 1;
        const int vq = L & 15, vb = L >> 4;
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (lq == vq && (j >> lg_jpb) == vb) scr[(16 * j + 4 * g + r) - vb * R] = t[j][qb][r];
        const float v1 = __shfl(cs[qb][0] + cs[qb][1], L, 64);
        const float v2 = __shfl(cs[qb][2] + cs[qb][3], L, 64);
        wave_sync_lds();
        if (lane == 0) {
          const int q = qw + 16 * qb + vq;
          const EecResult res = eec_locate<float>(scr, 1, R, v1, v2, fd.e_rel, fd.tn_s);
          int idx = -1;
          float nv = 0.f;
          if (res.status == EEC_LOCATED) {
            idx = res.index;
            const int key = key0 + vb * R + idx;
            const float old = scr[idx];
            int action = ABFT_ACT_RECOMPUTE;
            if (fd.recompute) {
              float acc = 0.f;
              for (int dd = 0; dd < D; ++dd)
                acc = fmaf(bf2f(A[int64_t(q) * lda + dd]), bf2f(Bm[int64_t(key) * ldb + dd]), acc);
              nv = acc;
            } else {
              nv = fix_by_checksum<float>(scr, 1, R, idx, v1, res.d1, fd.tc, &action);
            }
            scr[idx] = nv;
            record_event(fd.report, op, b, h, q, key, classify(old, fd.tn_s), action, old);
          }
          if (res.status != EEC_CLEAN && vec_flagged<float>(scr, 1, R, v1, fd.e_rel))
            record_event(fd.report, op, b, h, q, key0 + vb * R, ABFT_KIND_NONE,
                         ABFT_ACT_UNCORRECTABLE, 0.f);
          scr[R] = __int_as_float(idx);
          scr[R + 1] = nv;
        }
        wave_sync_lds();
        const int idx = __float_as_int(scr[R]);
        const float nv = scr[R + 1];
        if (idx >= 0) {
          const int kl = vb * R + idx;
#pragma unroll
          for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (lane == vq + 16 * ((kl & 15) >> 2) && j == (kl >> 4) && r == (kl & 3))
                t[j][qb][r] = nv;
        }
        wave_sync_lds();
      }
    }
  }

  // injected faults of op (test-only) on a 128-key x 32-query fp32 tile
  __device__ static void inject_tile(floatx4 (&t)[8][2], const FusedBwdDesc& fd, int op, int b,
                                     int h, int qw, int key0, int lane) {
    for (int f = 0; f < fd.n_faults; ++f) {
      const abft_fault ft = fd.faults[f];
      if (ft.op != op || ft.b != b || ft.h != h) continue;
      const int qi = ft.row - qw, ki = ft.col - key0;
      if (qi < 0 || qi >= 32 || ki < 0 || ki >= FT) continue;
      // under the mask only the block-lower-triangular region is computed
      if (fd.causal && ft.col / fd.R > ft.row / fd.R) continue;
      const int oq = qi >> 4, olane = (qi & 15) + 16 * ((ki & 15) >> 2);
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (lane == olane && qb == oq && j == (ki >> 4) && r == (ki & 3))
              t[j][qb][r] = ft.mode == ABFT_FAULT_FLIP ? flip_f32(t[j][qb][r]) : ft.value;
    }
  }

  __device__ static void run(const FusedBwdDesc& fd, char* smem) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lq = lane & 15, g = lane >> 4;
    const int S = fd.S, H = fd.H, R = fd.R, NB = FT / R, nqR = S / R;
    const int nqt = S / FT, nbh = fd.B * fd.nh;
    const int z = blockIdx.x % nbh;
    const int qt = fd.causal ? nqt - 1 - int(blockIdx.x) / nbh : int(blockIdx.x) / nbh;
    const int b = z / fd.nh, h = z % fd.nh;
    const int q0 = qt * FT, qw = q0 + wave * 32;
    const int64_t ld = 3 * int64_t(H);
    const bf16_t* base = static_cast<const bf16_t*>(fd.qkv) + int64_t(b) * S * ld;
    const bf16_t* Qp = base + h * D;
    const bf16_t* Kp = base + H + h * D;
    const bf16_t* Vp = base + 2 * H + h * D;
    const bf16_t* dCLp = static_cast<const bf16_t*>(fd.dcl) + int64_t(b) * S * H + h * D;
    const bf16_t* CLp = static_cast<const bf16_t*>(fd.cl) + int64_t(b) * S * H + h * D;
    const int nkt = fd.causal ? qt + 1 : nqt;
    const float sl2 = fd.scale * 1.4426950408889634f;
    const int lg_jpb = __builtin_ctz(R / 16);
    constexpr bool chk = CHK;

    // the statistics and the softmax backward's row term D = dCL . CL of
    // the lane's queries
    float mq[2], il[2], dq[2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int q = qw + 16 * qb + lq;
      float acc = 0.f;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const bf16x8 gv = *reinterpret_cast<const bf16x8*>(dCLp + int64_t(q) * H + 32 * kk + 8 * g);
        const bf16x8 cv = *reinterpret_cast<const bf16x8*>(CLp + int64_t(q) * H + 32 * kk + 8 * g);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = fmaf(float(gv[e]), float(cv[e]), acc);
      }
      dq[qb] = group4_sum(acc);
      const float* st = fd.stats + ((int64_t(b) * fd.nh + h) * S + q) * 2;
      mq[qb] = st[0];
      il[qb] = 1.f / st[1];
    }
    // Q and dCL images of the workgroup's queries (complete with tile 0)
#pragma unroll
    for (int hf = 0; hf < KH; ++hf) {
      DK::issue(Qp, ld, q0, S, hf * 64, smem + OFF_Q + hf * DK::BYTES, wave, lane);
      DK::issue(dCLp, H, q0, S, hf * 64, smem + OFF_G + hf * DK::BYTES, wave, lane);
    }

    float kcv[4] = {0.f, 0.f, 0.f, 0.f}, vcv[4] = {0.f, 0.f, 0.f, 0.f}, krv = 0.f;
    auto issue = [&](int kt) {
      const int key0 = kt * FT;
#pragma unroll
      for (int hf = 0; hf < KH; ++hf) {
        DK::issue(Kp, ld, key0, S, hf * 64, smem + hf * DK::BYTES, wave, lane);
        DK::issue(Vp, ld, key0, S, hf * 64, smem + OFF_V + hf * DK::BYTES, wave, lane);
      }
      if (chk) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const int e = tid + p * FNT;
          const int ee = e < NB * 2 * D ? e : 0;
          const int blk = ee / (2 * D), c = (ee / D) & 1, dd = ee % D;
          const float* row =
              fd.qkvc + ((int64_t(b) * nqR + key0 / R + blk) * 2 + c) * ld + h * D + dd;
          kcv[p] = row[H];
          vcv[p] = row[2 * H];
        }
        krv = fd.kr[((int64_t(b) * S + key0 + (tid >> 1)) * fd.nh + h) * 2 + (tid & 1)];
      }
    };
    auto commit = [&]() {
      if (chk) {
        bf16_t* kcs = reinterpret_cast<bf16_t*>(smem + OFF_KC);
        bf16_t* vcs = reinterpret_cast<bf16_t*>(smem + OFF_VC);
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const int e = tid + p * FNT;
          if (e < NB * 2 * D) {
            const int blk = e / (2 * D), c = (e / D) & 1, dd = e % D;
            const int r = (4 * blk + 2 * c) * SCL + dd;
            kcs[r] = f2bf(kcv[p]);
            kcs[r + SCL] = f2bf(kcv[p] - bf2f(f2bf(kcv[p])));
            vcs[r] = f2bf(vcv[p]);
            vcs[r + SCL] = f2bf(vcv[p] - bf2f(f2bf(vcv[p])));
          }
        }
        bf16_t* krs = reinterpret_cast<bf16_t*>(smem + OFF_KR);
        krs[(tid >> 1) * 16 + 2 * (tid & 1)] = f2bf(krv);
        krs[(tid >> 1) * 16 + 2 * (tid & 1) + 1] = f2bf(krv - bf2f(f2bf(krv)));
      }
    };
    // K^r strip: columns 0..3 per key (hi/lo of the sum and of the 1-based
    // weighted sum over the head dims, written with each tile); 4..15 zero
    bf16_t* krs = reinterpret_cast<bf16_t*>(smem + OFF_KR);
    if (chk)
      for (int e = tid; e < FT * 12; e += FNT) krs[(e / 12) * 16 + 4 + e % 12] = 0;

    floatx4 dqa[DB][2], kra[2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
      for (int db = 0; db < DB; ++db) dqa[db][qb] = floatx4{0.f, 0.f, 0.f, 0.f};
      kra[qb] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    float* scr = reinterpret_cast<float*>(smem + OFF_SCR) + wave * SCR;
    bf16_t* AP = static_cast<bf16_t*>(fd.ap) + (int64_t(b) * fd.nh + h) * S * S;
    bf16_t* dAS = static_cast<bf16_t*>(fd.das) + (int64_t(b) * fd.nh + h) * S * S;
    float* APr = fd.apr + (int64_t(b) * fd.nh + h) * S * nqR * 2;
    float* dASr = fd.dasr + (int64_t(b) * fd.nh + h) * S * nqR * 2;

    for (int kt = 0; kt < nkt; ++kt) {
      issue(kt);
      wait_vmcnt<0>();
      commit();
      __syncthreads();  // tile kt in LDS
      const int key0 = kt * FT;

      const bool diag = fd.causal && kt == qt;
      // B operand fragments of the wave's queries (rows of the Q or dCL image)
      auto bfrag = [&](int off, int qb, int kk) {
        return DK::frag(smem + off + (kk >> 1) * DK::BYTES, wave * 32 + 16 * qb, (kk & 1) * 32, lane);
      };
      // P^T, then dS^T, packed to bf16: pk[j][qb] holds keys 16 j + 4 g + 0..3
      // of query 16 qb + lane % 16
      uint2 pk[8][2];
      {
        // S^T = K Q^T with its strip rows, checked; P from the statistics
        floatx4 s[8][2], ks[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
          for (int j = 0; j < 8; ++j) s[j][qb] = floatx4{0.f, 0.f, 0.f, 0.f};
          ks[qb] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          const bf16x8 qf0 = bfrag(OFF_Q, 0, kk), qf1 = bfrag(OFF_Q, 1, kk);
          const char* sk = smem + (kk >> 1) * DK::BYTES;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const bf16x8 kf = DK::frag(sk, 16 * j, (kk & 1) * 32, lane);
            s[j][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf0, s[j][0], 0, 0, 0);
            s[j][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf1, s[j][1], 0, 0, 0);
          }
          if (chk) {
            const bf16_t* kcs = reinterpret_cast<const bf16_t*>(smem + OFF_KC);
            const bf16x8 kc = *reinterpret_cast<const bf16x8*>(kcs + lq * SCL + 32 * kk + 8 * g);
            ks[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kc, qf0, ks[0], 0, 0, 0);
            ks[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kc, qf1, ks[1], 0, 0, 0);
          }
        }
        if (fd.n_faults > 0) inject_tile(s, fd, ABFT_OP_AS, b, h, qw, key0, lane);
        if (chk) check_tile(s, ks, fd, ABFT_OP_AS, b, h, qw, key0, Qp, Kp, ld, ld, scr, lane);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          const int q = qw + 16 * qb + lq;
          float a1[4] = {0.f, 0.f, 0.f, 0.f}, a2[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            float a[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool live = !(diag && key0 + 16 * j + 4 * g + r > q);
              a[r] = live ? bf2f(f2bf(__builtin_amdgcn_exp2f(s[j][qb][r] * sl2 - mq[qb]) * il[qb]))
                          : 0.f;
            }
            pk[j][qb] = uint2{pack2(a[0], a[1]), pack2(a[2], a[3])};
            *reinterpret_cast<uint2*>(AP + int64_t(q) * S + key0 + 16 * j + 4 * g) = pk[j][qb];
            if (!chk) continue;
            // the 16-key group j lies in block j >> lg_jpb; weights 1..R in it
            const int wb = ((16 * j) & (R - 1)) + 4 * g + 1;
            const float sa1 = (a[0] + a[1]) + (a[2] + a[3]);
            const float sa2 = float(wb) * a[0] + float(wb + 1) * a[1] + float(wb + 2) * a[2] +
                              float(wb + 3) * a[3];
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if ((j >> lg_jpb) == i) { a1[i] += sa1; a2[i] += sa2; }
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (chk && i < NB) {
              const float t1 = group4_sum(a1[i]), t2 = group4_sum(a2[i]);
              if (g == i) {
                const int64_t o = (int64_t(q) * nqR + key0 / R + i) * 2;
                APr[o] = t1;
                APr[o + 1] = t2;
              }
            }
          }
        }
      }
      {
        // dP^T = V dCL^T with its strip rows, checked; dS from P and dP
        floatx4 dp[8][2], vs[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
          for (int j = 0; j < 8; ++j) dp[j][qb] = floatx4{0.f, 0.f, 0.f, 0.f};
          vs[qb] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          const bf16x8 gf0 = bfrag(OFF_G, 0, kk), gf1 = bfrag(OFF_G, 1, kk);
          const char* sv = smem + OFF_V + (kk >> 1) * DK::BYTES;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const bf16x8 vf = DK::frag(sv, 16 * j, (kk & 1) * 32, lane);
            dp[j][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, gf0, dp[j][0], 0, 0, 0);
            dp[j][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, gf1, dp[j][1], 0, 0, 0);
          }
          if (chk) {
            const bf16_t* vcs = reinterpret_cast<const bf16_t*>(smem + OFF_VC);
            const bf16x8 vc = *reinterpret_cast<const bf16x8*>(vcs + lq * SCL + 32 * kk + 8 * g);
            vs[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vc, gf0, vs[0], 0, 0, 0);
            vs[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vc, gf1, vs[1], 0, 0, 0);
          }
        }
        if (fd.n_faults > 0) inject_tile(dp, fd, ABFT_OP_DAP, b, h, qw, key0, lane);
        if (chk) check_tile(dp, vs, fd, ABFT_OP_DAP, b, h, qw, key0, dCLp, Vp, H, ld, scr, lane);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          const int q = qw + 16 * qb + lq;
          float d1[4] = {0.f, 0.f, 0.f, 0.f}, d2[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float a[4] = {__uint_as_float(pk[j][qb].x << 16),
                                __uint_as_float(pk[j][qb].x & 0xffff0000u),
                                __uint_as_float(pk[j][qb].y << 16),
                                __uint_as_float(pk[j][qb].y & 0xffff0000u)};
            float ds[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool live = !(diag && key0 + 16 * j + 4 * g + r > q);
              ds[r] = live ? bf2f(f2bf(fd.scale * a[r] * (dp[j][qb][r] - dq[qb]))) : 0.f;
            }
            pk[j][qb] = uint2{pack2(ds[0], ds[1]), pack2(ds[2], ds[3])};
            *reinterpret_cast<uint2*>(dAS + int64_t(q) * S + key0 + 16 * j + 4 * g) = pk[j][qb];
            if (!chk) continue;
            const int wb = ((16 * j) & (R - 1)) + 4 * g + 1;
            const float sd1 = (ds[0] + ds[1]) + (ds[2] + ds[3]);
            const float sd2 = float(wb) * ds[0] + float(wb + 1) * ds[1] + float(wb + 2) * ds[2] +
                              float(wb + 3) * ds[3];
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if ((j >> lg_jpb) == i) { d1[i] += sd1; d2[i] += sd2; }
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (chk && i < NB) {
              const float u1 = group4_sum(d1[i]), u2 = group4_sum(d2[i]);
              if (g == i) {
                const int64_t o = (int64_t(q) * nqR + key0 / R + i) * 2;
                dASr[o] = u1;
                dASr[o + 1] = u2;
              }
            }
          }
        }
      }

      // dQ^T += K^T dS^T and (dQ^r)^T += (K^r)^T dS^T
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        bf16x8 pf[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          const uint4 u = {pk[2 * t][qb].x, pk[2 * t][qb].y, pk[2 * t + 1][qb].x,
                           pk[2 * t + 1][qb].y};
          pf[qb] = __builtin_bit_cast(bf16x8, u);
        }
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          TrPair kp = kt_frag(smem, 16 * db, 32 * t, lane);
          const bf16x8 kf = tr_join(kp);
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
            dqa[db][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, pf[qb], dqa[db][qb], 0, 0, 0);
        }
        if (chk) {
          TrPair rp = kr_frag(krs, 32 * t, lane);
          const bf16x8 rf = tr_join(rp);
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
            kra[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rf, pf[qb], kra[qb], 0, 0, 0);
        }
      }
      __syncthreads();  // the one stage is reloaded next
    }

    // dQ: round, check against dQ^r, store
    bf16_t* dQp = static_cast<bf16_t*>(fd.dq) + int64_t(b) * S * fd.ldq + h * D;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int q = qw + 16 * qb + lq;
      float ov[DB][4];
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 4; ++r) ov[db][r] = bf2f(f2bf(dqa[db][qb][r]));
      if (fd.n_faults > 0) {
        for (int f = 0; f < fd.n_faults; ++f) {
          const abft_fault ft = fd.faults[f];
          if (ft.op != ABFT_OP_DQ || ft.b != b || ft.h != h || ft.row != q) continue;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (ft.col == 16 * db + 4 * g + r)
                ov[db][r] = ft.mode == ABFT_FAULT_FLIP ? bf2f(flip_exponent_msb(f2bf(ov[db][r])))
                                                       : bf2f(f2bf(ft.value));
        }
      }
      if (chk) {
        const float c1 = __shfl(kra[qb][0] + kra[qb][1], lq, 64);
        const float c2 = __shfl(kra[qb][2] + kra[qb][3], lq, 64);
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
          if (lane == 0) {
            const int qq = qw + 16 * qb + L;
            const EecResult res = eec_locate<float>(scr, 1, D, v1, v2, fd.e_rel, fd.tn);
            int idx = -1;
            float nv = 0.f;
            if (res.status == EEC_LOCATED) {
              idx = res.index;
              const float old = scr[idx];
              int action = 0;
              nv = bf2f(f2bf(fix_by_checksum<float>(scr, 1, D, idx, v1, res.d1, fd.tc, &action)));
              scr[idx] = nv;
              record_event(fd.report, ABFT_OP_DQ, b, h, qq, idx, classify(old, fd.tn), action, old);
            }
            if (res.status != EEC_CLEAN && vec_flagged<float>(scr, 1, D, v1, fd.e_rel))
              record_event(fd.report, ABFT_OP_DQ, b, h, qq, 0, ABFT_KIND_NONE,
                           ABFT_ACT_UNCORRECTABLE, 0.f);
            scr[D] = __int_as_float(idx);
            scr[D + 1] = nv;
          }
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
        *reinterpret_cast<uint2*>(dQp + int64_t(q) * fd.ldq + 16 * db + 4 * g) = w;
      }
    }
  }
};

// one wave per SIMD for the checked kernels: their registers fit without
// spills (two waves per SIMD spilled and ran slower)
template <int D, bool CHK>
__global__ __launch_bounds__(FNT) __attribute__((amdgpu_waves_per_eu(D == 64 && !CHK ? 2 : 1)))
void fused_bwd_kernel(FusedBwdDesc fd) {
  extern __shared__ __align__(16) char smem[];
  FusedBwd<D, CHK>::run(fd, smem);
}

template <int D, bool PROT>
__global__ __launch_bounds__(FNT) __attribute__((amdgpu_waves_per_eu(2)))
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
  hipLaunchKernelGGL(kern, dim3(unsigned(grid)), dim3(FNT), F::LDS_BYTES, s, fd);
  return hipGetLastError();
}

template <int D, bool CHK>
hipError_t launch_bwd_d(const FusedBwdDesc& fd, hipStream_t s) {
  using F = FusedBwd<D, CHK>;
  static bool attr = false;
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(fused_bwd_kernel<D, CHK>),
        hipFuncAttributeMaxDynamicSharedMemorySize, F::LDS_BYTES);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int64_t grid = int64_t(fd.B) * fd.nh * (fd.S / FT);
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL((fused_bwd_kernel<D, CHK>), dim3(unsigned(grid)), dim3(FNT), F::LDS_BYTES, s,
                     fd);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_fused_bwd(const FusedBwdDesc& fd, hipStream_t s) {
  if (fd.S % FT != 0 || fd.R < 32 || FT % fd.R != 0 || fd.H != fd.nh * fd.D ||
      fd.qkv == nullptr || fd.cl == nullptr || fd.dcl == nullptr || fd.stats == nullptr ||
      fd.ap == nullptr || fd.apr == nullptr || fd.das == nullptr || fd.dasr == nullptr ||
      fd.dq == nullptr || fd.ldq < fd.H || (fd.check && (fd.qkvc == nullptr || fd.kr == nullptr)))
    return hipErrorInvalidValue;
  if (fd.D == 64) return fd.check ? launch_bwd_d<64, true>(fd, s) : launch_bwd_d<64, false>(fd, s);
  if (fd.D == 128) return fd.check ? launch_bwd_d<128, true>(fd, s) : launch_bwd_d<128, false>(fd, s);
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
