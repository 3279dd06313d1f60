// Device-side helpers: storage conversions, EEC-ABFT on one vector, event
// recording. Included by the kernel translation units only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_abft.h"

namespace abft {

typedef uint16_t bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// float -> bfloat16, round to nearest even (gfx950 converts in hardware,
// v_cvt_pk_bf16_f32; NaN stays a quiet NaN, overflow becomes INF).
__device__ __forceinline__ bf16_t f2bf(float f) {
  return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f));
}

// The fault injector's bit flip: the most significant exponent bit of a
// stored value (bit 14 of bf16, bit 30 of fp32).
__device__ __forceinline__ bf16_t flip_exponent_msb(bf16_t v) { return bf16_t(v ^ 0x4000u); }
__device__ __forceinline__ float flip_exponent_msb(float v) {
  return __uint_as_float(__float_as_uint(v) ^ 0x40000000u);
}

template <class T> struct Storage;
template <> struct Storage<bf16_t> {
  __device__ static float load(bf16_t v) { return bf2f(v); }
  __device__ static bf16_t store(float f) { return f2bf(f); }
  __device__ static float round(float f) { return bf2f(f2bf(f)); }
};
template <> struct Storage<float> {
  __device__ static float load(float v) { return v; }
  __device__ static float store(float f) { return f; }
  __device__ static float round(float f) { return f; }
};

__device__ __forceinline__ bool is_finite(float x) {
  return (__float_as_uint(x) & 0x7f800000u) != 0x7f800000u;
}
__device__ __forceinline__ bool is_nan(float x) {
  return (__float_as_uint(x) & 0x7fffffffu) > 0x7f800000u;
}
__device__ __forceinline__ bool is_inf(float x) {
  return (__float_as_uint(x) & 0x7fffffffu) == 0x7f800000u;
}

// Extreme-value class of a stored value (paper Sec. 2.2); tn is the
// near-INF threshold as stored.
__device__ __forceinline__ int classify(float v, float tn) {
  if (is_nan(v)) return ABFT_KIND_NAN;
  if (is_inf(v)) return ABFT_KIND_INF;
  if (fabsf(v) >= tn) return ABFT_KIND_NEAR_INF;
  return ABFT_KIND_NUMERIC;
}

// Detection rule (Sec. 2.3): flagged unless d1 is finite and |d1| <= E,
// E = e_rel * sum|v| over finite v (+ a tiny floor).
__device__ __forceinline__ bool flagged(float d1, float abs_sum, float e_rel) {
  const float E = e_rel * abs_sum + 1e-30f;
  return !(is_finite(d1) && fabsf(d1) <= E);
}

enum { EEC_CLEAN = 0, EEC_LOCATED = 1, EEC_PROPAGATED = 2 };
struct EecResult {
  int status;
  int index;
  float d1;
};

// EEC-ABFT on one vector of n stored values v[k * stride] (Sec. 4.2 cases
// 1-4 with the mixed-type candidate sets of Sec. 4.3). c1, c2: propagated
// unweighted and weighted (1-based weights) checksums.
template <class T, int UNR = 8>
__device__ EecResult eec_locate(const T* v, int stride, int n, float c1, float c2, float e_rel,
                                float tn) {
  float r1 = 0.f, r2 = 0.f, sa = 0.f;
  // (unrolled UNR ways: the loads of a rare path go out together instead
  // of one memory latency each; callers short of registers keep UNR = 1,
  // since the unrolled copy's registers count against the caller's)
#pragma unroll UNR
  for (int k = 0; k < n; ++k) {
    const float x = Storage<T>::load(v[k * stride]);
    r1 += x;
    r2 += float(k + 1) * x;
    sa += is_finite(x) ? fabsf(x) : 0.f;
  }
  const float d1 = c1 - r1, d2 = c2 - r2;
  EecResult res{EEC_CLEAN, -1, d1};
  if (!flagged(d1, sa, e_rel)) return res;
  const int mode = is_finite(d1) ? 1 : (is_inf(d1) ? 2 : 3);
  // candidates counted with selects (straight-line code: a branch per
  // element turns the unrolled loop into nested divergent loops)
  const bool any_inf = mode == 2, any_nonfin = mode == 3;
  int cnt = 0, idx = -1;
#pragma unroll UNR
  for (int k = 0; k < n; ++k) {
    const float x = Storage<T>::load(v[k * stride]);
    const bool fin = is_finite(x);
    const bool nearv = fin && fabsf(x) >= tn;
    const bool cand = nearv || (any_inf && is_inf(x)) || (any_nonfin && !fin);
    cnt += cand ? 1 : 0;
    idx = cand ? k : idx;
  }
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

// Correction from the checksums alone (Sec. 4.2): DELTA when |d1| <=
// t_correct, otherwise RECONSTRUCT v_i = c1 - sum_{k != i} v_k.
template <class T, int UNR = 8>
__device__ float fix_by_checksum(const T* v, int stride, int n, int i, float c1, float d1,
                                 float tc, int* action) {
  if (is_finite(d1) && fabsf(d1) <= tc) {
    *action = ABFT_ACT_DELTA;
    return Storage<T>::load(v[i * stride]) + d1;
  }
  float s = 0.f;
#pragma unroll UNR
  for (int k = 0; k < n; ++k) {
    const float x = Storage<T>::load(v[k * stride]);
    s += k != i ? x : 0.f;
  }
  *action = ABFT_ACT_RECONSTRUCT;
  return c1 - s;
}

// Unweighted and weighted sums of a vector (checksum refresh, Sec. 4.3).
template <class T>
__device__ void vec_checksums(const T* v, int stride, int n, float* c1, float* c2) {
  float r1 = 0.f, r2 = 0.f;
#pragma unroll 8
  for (int k = 0; k < n; ++k) {
    const float x = Storage<T>::load(v[k * stride]);
    r1 += x;
    r2 += float(k + 1) * x;
  }
  *c1 = r1;
  *c2 = r2;
}

// Detection only. The magnitude sum may include non-finite elements: any
// INF or NaN makes r1, hence d1, non-finite, which is flagged whatever E is,
// so the decision equals the rule with E over finite elements.
template <class T>
__device__ bool vec_flagged(const T* v, int stride, int n, float c1, float e_rel) {
  float r1 = 0.f, sa = 0.f;
#pragma unroll 8
  for (int k = 0; k < n; ++k) {
    const float x = Storage<T>::load(v[k * stride]);
    r1 += x;
    sa += fabsf(x);
  }
  return flagged(c1 - r1, sa, e_rel);
}

// Cross-lane sums on DPP moves (no LDS round trip). After group_sum<W>
// every lane of an aligned group of W lanes holds the same value: each
// step adds a value and its partner's, so both partners get the same sum.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}
constexpr int DPP_XOR1 = 0xb1;         // quad_perm [1,0,3,2]
constexpr int DPP_XOR2 = 0x4e;         // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141; // lane i <- lane 7 - i within 8
constexpr int DPP_MIRROR = 0x140;      // lane i <- lane 15 - i within 16

template <int W>
__device__ __forceinline__ float group_sum(float x) {
  if constexpr (W >= 2) x += dpp_mov<DPP_XOR1>(x);
  if constexpr (W >= 4) x += dpp_mov<DPP_XOR2>(x);
  if constexpr (W >= 8) x += dpp_mov<DPP_HALF_MIRROR>(x);
  if constexpr (W >= 16) x += dpp_mov<DPP_MIRROR>(x);
  if constexpr (W >= 32) x += __shfl_xor(x, 16, 64);
  if constexpr (W >= 64) x += __shfl_xor(x, 32, 64);
  return x;
}
// group_sum for a wave-uniform runtime width (a power of two <= 64)
__device__ __forceinline__ float group_sum_n(float x, int w) {
  switch (w) {
    case 1: return x;
    case 2: return group_sum<2>(x);
    case 4: return group_sum<4>(x);
    case 8: return group_sum<8>(x);
    case 16: return group_sum<16>(x);
    case 32: return group_sum<32>(x);
    default: return group_sum<64>(x);
  }
}

__device__ inline void record_event(abft_report* rep, int op, int b, int h, int row, int col,
                                    int kind, int action, float observed) {
  if (rep == nullptr) return;
  const int slot = atomicAdd(&rep->n_events, 1);
  if (action == ABFT_ACT_UNCORRECTABLE)
    atomicAdd(&rep->n_uncorrectable, 1);
  else
    atomicAdd(&rep->n_corrected, 1);
  if (slot < rep->capacity) {
    abft_event* e = &rep->events[slot];
    e->op = op;
    e->b = b;
    e->h = h;
    e->row = row;
    e->col = col;
    e->kind = kind;
    e->action = action;
    e->reserved = 0;
    e->observed = observed;
    e->reserved2 = 0.f;
  } else {
    atomicOr(&rep->overflow, 1);
  }
}

}  // namespace abft
