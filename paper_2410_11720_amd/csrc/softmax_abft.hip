// Softmax over keys with checksum carry-through, forward and backward.
//
// The softmax itself is not ABFT-protected (paper Sec. 4.4 protects the
// GEMMs); what it does for ABFT is encode its output on the fly: the
// column checksums of AP over each R-row query block feed CL^c = AP^c V
// (the S_CL section encodes AP with column checksums, Sec. 4.4), and the
// row checksums of AP over each R-column key block feed the checksum of
// dV = AP^T dCL in the backward. The backward kernel does the same for
// dAS (feeding dQ = dAS K and dK = dAS^T Q).
//
// One workgroup owns one query block of R rows of one (batch, head); each
// wave walks its rows; a lane owns 16-byte chunks of columns, so every row
// is read and written with fully coalesced vector accesses and the column
// checksums accumulate in registers. Masked entries (key > query under a
// causal mask) are selected to zero; keys past the end of the score tile
// that holds the diagonal are neither read nor written.
#include "abft_internal.hpp"
#include "abft_device.hpp"

namespace abft {
namespace {

constexpr int NT = 256;

template <class T> struct Vec;
template <> struct Vec<bf16_t> {
  static constexpr int N = 8;
  __device__ static void load(const bf16_t* p, float* out) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      out[2 * q] = __uint_as_float(w[q] << 16);
      out[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
    }
  }
  __device__ static void store(bf16_t* p, const float* in) {
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) w[q] = uint32_t(f2bf(in[2 * q])) | (uint32_t(f2bf(in[2 * q + 1])) << 16);
    *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
  }
};
template <> struct Vec<float> {
  static constexpr int N = 4;
  __device__ static void load(const float* p, float* out) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
  }
  __device__ static void store(float* p, const float* in) {
    *reinterpret_cast<float4*>(p) = make_float4(in[0], in[1], in[2], in[3]);
  }
};

__device__ __forceinline__ float nanmax(float a, float b) {  // NaN-propagating max
  return (is_nan(a) || a > b) ? a : b;
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = nanmax(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
// sum over aligned groups of `width` lanes (width a power of two <= 64)
__device__ __forceinline__ float group_sum(float x, int width) {
  for (int o = 1; o < width; o <<= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// CH: 16-byte chunks per lane per row (S <= 64 * CH * VEC); RPI rows per
// iteration per wave; PF: prefetch the next iteration's rows.
template <class T, int CH, bool BWD, int RPI, bool PF>
__global__ __launch_bounds__(NT) void softmax_kernel(SoftmaxDesc d) {
  constexpr int V = Vec<T>::N;
  extern __shared__ __align__(16) char smem[];
  float* colacc = reinterpret_cast<float*>(smem);  // [S][2]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int qb = blockIdx.x, z = blockIdx.y;
  const int S = d.S, R = d.R;
  const int nq = S / R;
  const int s_valid =
      d.causal ? min(S, ((qb + 1) * R + d.kv_align - 1) / d.kv_align * d.kv_align) : S;
  const int64_t mat = int64_t(z) * S * S;
  const T* src = static_cast<const T*>(BWD ? d.AP : d.AS) + mat;
  const T* src2 = BWD ? static_cast<const T*>(d.dAP) + mat : nullptr;
  T* dst = static_cast<T*>(BWD ? d.dAS : d.AP) + mat;
  const int lanes_per_kb = R / V;  // lanes covering one key block

  float c1[CH][V], c2[CH][V];
#pragma unroll
  for (int t = 0; t < CH; ++t)
#pragma unroll
    for (int e = 0; e < V; ++e) c1[t][e] = c2[t][e] = 0.f;

  const float l2e = 1.4426950408889634f;
  // Rows of this wave: rl = wave + 4 * (it * RPI + u), u < RPI. With PF the
  // loads of iteration it + 1 are issued before iteration it is computed
  // (two register buffers, the loop unrolled by two so that buffer indices
  // stay compile-time constants).
  auto load_rows = [&](float (&x)[RPI][CH][V], float (&y)[RPI][CH][V], int it) {
#pragma unroll
    for (int u = 0; u < RPI; ++u) {
      const int i = qb * R + wave + 4 * (it * RPI + u);
#pragma unroll
      for (int t = 0; t < CH; ++t) {
        const int j0 = (lane + 64 * t) * V;
        if (j0 < s_valid) {
          Vec<T>::load(src + int64_t(i) * S + j0, x[u][t]);
          if (BWD) Vec<T>::load(src2 + int64_t(i) * S + j0, y[u][t]);
        } else {
#pragma unroll
          for (int e = 0; e < V; ++e) x[u][t][e] = y[u][t][e] = 0.f;
        }
      }
    }
  };
  auto process_rows = [&](float (&xr)[RPI][CH][V], float (&yr)[RPI][CH][V], int it) {
#pragma unroll
    for (int u = 0; u < RPI; ++u) {
      const int rl = wave + 4 * (it * RPI + u);
      const int i = qb * R + rl;
      float (&x)[CH][V] = xr[u];
      float (&y)[CH][V] = yr[u];
      if (!BWD) {
        // AP = softmax(scale * AS) over unmasked keys, in base 2
        const float sc = d.scale * l2e;
        float mx = -INFINITY;
#pragma unroll
        for (int t = 0; t < CH; ++t)
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const int j = (lane + 64 * t) * V + e;
            const bool live = j < s_valid && (!d.causal || j <= i);
            x[t][e] = live ? x[t][e] * sc : -INFINITY;
            mx = nanmax(mx, x[t][e]);
          }
        mx = wave_max(mx);
        float sum = 0.f;
#pragma unroll
        for (int t = 0; t < CH; ++t)
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const int j = (lane + 64 * t) * V + e;
            const bool live = j < s_valid && (!d.causal || j <= i);
            const float ev = live ? __builtin_amdgcn_exp2f(x[t][e] - mx) : 0.f;
            x[t][e] = ev;
            sum += ev;
          }
        sum = wave_sum(sum);
        const float inv = 1.f / sum;
#pragma unroll
        for (int t = 0; t < CH; ++t)
#pragma unroll
          for (int e = 0; e < V; ++e) x[t][e] = Storage<T>::round(x[t][e] * inv);
      } else {
        // dAS = scale * AP * (dAP - D), D = sum_j AP_j dAP_j over unmasked keys
        float dot = 0.f;
#pragma unroll
        for (int t = 0; t < CH; ++t)
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const int j = (lane + 64 * t) * V + e;
            const bool live = j < s_valid && (!d.causal || j <= i);
            dot += live ? x[t][e] * y[t][e] : 0.f;
          }
        dot = wave_sum(dot);
#pragma unroll
        for (int t = 0; t < CH; ++t)
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const int j = (lane + 64 * t) * V + e;
            const bool live = j < s_valid && (!d.causal || j <= i);
            x[t][e] = live ? Storage<T>::round(d.scale * x[t][e] * (y[t][e] - dot)) : 0.f;
          }
      }
      // store, accumulate column checksums, emit row checksums per key block
      const float wr = float(rl + 1);
#pragma unroll
      for (int t = 0; t < CH; ++t) {
        const int j0 = (lane + 64 * t) * V;
        float r1 = 0.f, r2 = 0.f;
        if (j0 < s_valid) {
          Vec<T>::store(dst + int64_t(i) * S + j0, x[t]);
#pragma unroll
          for (int e = 0; e < V; ++e) {
            c1[t][e] += x[t][e];
            c2[t][e] += wr * x[t][e];
            r1 += x[t][e];
            r2 += float(((j0 + e) & (R - 1)) + 1) * x[t][e];
          }
        }
        if (d.row_chk != nullptr && (64 * t * V) < s_valid) {
          r1 = group_sum(r1, lanes_per_kb);
          r2 = group_sum(r2, lanes_per_kb);
          const int kb = j0 / R;
          if ((lane % lanes_per_kb) == 0 && j0 < s_valid) {
            float* rc = d.row_chk + ((int64_t(z) * S + i) * nq + kb) * 2;
            rc[0] = r1;
            rc[1] = r2;
          }
        }
      }
    }
  };

  const int n_it = R / (4 * RPI);
  float xa[RPI][CH][V], ya[RPI][CH][V];
  if constexpr (PF) {
    float xb[RPI][CH][V], yb[RPI][CH][V];
    load_rows(xa, ya, 0);
    for (int it = 0; it < n_it; it += 2) {
      if (it + 1 < n_it) load_rows(xb, yb, it + 1);
      process_rows(xa, ya, it);
      if (it + 2 < n_it) load_rows(xa, ya, it + 2);
      if (it + 1 < n_it) process_rows(xb, yb, it + 1);
    }
  } else {
    for (int it = 0; it < n_it; ++it) {
      load_rows(xa, ya, it);
      process_rows(xa, ya, it);
    }
  }

  // combine the four waves' column checksums in a fixed order
  if (d.col_chk != nullptr) {
    for (int w = 0; w < 4; ++w) {
      if (wave == w) {
#pragma unroll
        for (int t = 0; t < CH; ++t)
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const int j = (lane + 64 * t) * V + e;
            if (j < s_valid) {
              if (w == 0) {
                colacc[2 * j] = c1[t][e];
                colacc[2 * j + 1] = c2[t][e];
              } else {
                colacc[2 * j] += c1[t][e];
                colacc[2 * j + 1] += c2[t][e];
              }
            }
          }
      }
      __syncthreads();
    }
    float* cc = d.col_chk + (int64_t(z) * nq + qb) * 2 * S;
    for (int j = tid; j < s_valid; j += NT) {
      cc[j] = colacc[2 * j];
      cc[S + j] = colacc[2 * j + 1];
    }
  }
}

template <bool BWD>
hipError_t launch_sm(const SoftmaxDesc& d, int dtype, hipStream_t s) {
  const int V = dtype == ABFT_FP32 ? 4 : 8;
  const int ch = (d.S + 64 * V - 1) / (64 * V);
  dim3 grid(d.S / d.R, d.B * d.nh);
  const size_t lds = size_t(d.S) * 2 * sizeof(float);
#define SM_CASE(TT, CHV)                                                                      \
  if (ch <= CHV) {                                                                            \
    auto k = softmax_kernel<TT, CHV, BWD, (CHV == 1 ? 2 : 1), (CHV <= 2)>;                    \
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),                       \
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)); \
    if (e != hipSuccess) return e;                                                            \
    hipLaunchKernelGGL(k, grid, dim3(NT), lds, s, d);                                         \
    return hipGetLastError();                                                                 \
  }
  if (dtype == ABFT_FP32) {
    SM_CASE(float, 1) SM_CASE(float, 2) SM_CASE(float, 4) SM_CASE(float, 8) SM_CASE(float, 16)
  } else {
    SM_CASE(bf16_t, 1) SM_CASE(bf16_t, 2) SM_CASE(bf16_t, 4) SM_CASE(bf16_t, 8)
  }
#undef SM_CASE
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_softmax_fwd(const SoftmaxDesc& d, int dtype, hipStream_t s) {
  return launch_sm<false>(d, dtype, s);
}
hipError_t launch_softmax_bwd(const SoftmaxDesc& d, int dtype, hipStream_t s) {
  return launch_sm<true>(d, dtype, s);
}

}  // namespace abft
