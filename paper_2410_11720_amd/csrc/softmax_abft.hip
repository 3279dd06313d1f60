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
#include <atomic>

#include "abft_internal.hpp"
#include "abft_device.hpp"

namespace abft {
namespace {

constexpr int NT = 256;

template <class T> struct Vec;
template <> struct Vec<bf16_t> {
  static constexpr int N = 8;
  __device__ static void unpack(const uint4& v, float* out) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      out[2 * q] = __uint_as_float(w[q] << 16);
      out[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
    }
  }
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
  __device__ static void unpack(const uint4& v, float* out) {
    out[0] = __uint_as_float(v.x); out[1] = __uint_as_float(v.y);
    out[2] = __uint_as_float(v.z); out[3] = __uint_as_float(v.w);
  }
  __device__ static void load(const float* p, float* out) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
  }
  __device__ static void store(float* p, const float* in) {
    *reinterpret_cast<float4*>(p) = make_float4(in[0], in[1], in[2], in[3]);
  }
};

__device__ __forceinline__ float lane_of(float x, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), l));
}
__device__ __forceinline__ float wave_sum(float x) {
  x = group_sum<16>(x);
  return (lane_of(x, 0) + lane_of(x, 16)) + (lane_of(x, 32) + lane_of(x, 48));
}
// Row maximum. fmaxf skips a NaN, but a NaN still reaches every output
// through the row sum (exp2 of NaN), exactly as a NaN-propagating maximum
// would make it.
__device__ __forceinline__ float wave_max(float x) {
  x = fmaxf(x, dpp_mov<DPP_XOR1>(x));
  x = fmaxf(x, dpp_mov<DPP_XOR2>(x));
  x = fmaxf(x, dpp_mov<DPP_HALF_MIRROR>(x));
  x = fmaxf(x, dpp_mov<DPP_MIRROR>(x));
  return fmaxf(fmaxf(lane_of(x, 0), lane_of(x, 16)), fmaxf(lane_of(x, 32), lane_of(x, 48)));
}
// row checksum pair of a key block spread over w lanes (w uniform)
__device__ __forceinline__ void kb_sums(float& r1, float& r2, int w) {
  r1 = group_sum_n(r1, w);
  r2 = group_sum_n(r2, w);
}

// Round a chunk to storage in place; `bits` receives the stored image.
__device__ __forceinline__ void round_chunk(float (&x)[8], uint4& bits) {
  uint32_t w[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    w[q] = uint32_t(f2bf(x[2 * q])) | (uint32_t(f2bf(x[2 * q + 1])) << 16);
    x[2 * q] = __uint_as_float(w[q] << 16);
    x[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
  }
  bits = make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ __forceinline__ void round_chunk(float (&x)[4], uint4& bits) {
  bits = make_uint4(__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]),
                    __float_as_uint(x[3]));
}

// CH: 16-byte chunks per lane per row (S <= 64 * CH * VEC); RPI rows per
// iteration per wave; PF: prefetch the next iteration's rows; CHK: encode
// the checksums (some of col_chk, row_chk given).
template <class T, int CH, bool BWD, int RPI, bool PF, bool CHK>
__global__ __launch_bounds__(NT) void softmax_kernel(SoftmaxDesc d) {
  constexpr int V = Vec<T>::N;
  extern __shared__ __align__(16) char smem[];
  float* colacc = reinterpret_cast<float*>(smem);  // [8][S]

  // the wave index is uniform over the wave: row indices and row
  // addresses stay in scalar registers
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // One-dimensional grid, (batch, head) fastest: consecutive workgroups go
  // to different XCDs, so every XCD gets whole heads and the same mix of
  // block costs; under a causal mask the cost order runs from the longest
  // query blocks to the shortest.
  const int S = d.S, R = d.R;
  const int nq = S / R, nbh = d.B * d.nh;
  // Under a causal mask block costs differ up to nq times, and at these
  // sizes the whole grid is resident at once: workgroups are dealt
  // round-robin to the 8 XCDs and then to the CUs of each XCD, so the CU
  // that takes arrival slot m of its XCD also takes slots m + n, m + 2n, ...
  // (n CUs per XCD). Taking the cost order forwards in even rounds and
  // backwards in odd ones (a snake deal) evens out the CUs' sums; the
  // remap swaps pairs of workgroups inside a round, so it is a bijection
  // for any grid.
  int bid = blockIdx.x;
  if (d.causal && d.xcd_cus > 0) {
    const int n = d.xcd_cus, x = bid & 7, m = bid >> 3, rd = m / n, c = m - rd * n;
    const int t = 8 * (rd * n + ((rd & 1) ? n - 1 - c : c)) + x;
    if (t < int(gridDim.x)) bid = t;
  }
  const int z = bid % nbh, r = bid / nbh;
  const int qb = d.causal ? nq - 1 - r : r;
  const int s_valid =
      d.causal ? min(S, ((qb + 1) * R + d.kv_align - 1) / d.kv_align * d.kv_align) : S;
  const int64_t mat = int64_t(z) * S * S;
  const T* src = static_cast<const T*>(BWD ? d.AP : d.AS) + mat;
  const T* src2 = BWD ? static_cast<const T*>(d.dAP) + mat : nullptr;
  T* dst = static_cast<T*>(BWD ? d.dAS : d.AP) + mat;
  const int lanes_per_kb = R / V;  // lanes covering one key block
  // bf16: lane l holds chunk lc = 4 (l % 16) + l / 16 of each 64-chunk run,
  // so that the A operand of a 16x16x32 MFMA over a run's stored chunks
  // has row m = 32-key quarter m of the run (lanes m, m+16, m+32, m+48 hold
  // its four chunks): the row checksums per key block come from one MFMA
  // per run against a constant [ones | in-quarter index] operand
  constexpr bool PERM = V == 8;
  const int lc = PERM ? (lane & 15) * 4 + (lane >> 4) : lane;
  bf16x8 bsum;
  if constexpr (PERM) {
    const int n = lane & 15, gk = lane >> 4;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      bsum[e] = __builtin_bit_cast(__bf16, f2bf(n == 0 ? 1.f : (n == 1 ? float(8 * gk + e) : 0.f)));
  }

  float c1[CH][V], c2[CH][V];
#pragma unroll
  for (int t = 0; t < CH; ++t)
#pragma unroll
    for (int e = 0; e < V; ++e) c1[t][e] = c2[t][e] = 0.f;

  const float l2e = 1.4426950408889634f;
  // Rows of this wave: rl = wave + 4 * (it * RPI + u), u < RPI. With PF the
  // loads of iteration it + 1 are issued once iteration it's loaded values
  // are unpacked, before it is computed (one register buffer).
  // Loads are unconditional (a chunk past s_valid, or under the causal
  // mask wholly past the diagonal, reads the row's chunk holding the
  // diagonal instead, an address another lane of the same load reads, and
  // lies past the live prefix that the arithmetic keeps), so every load of
  // an iteration is in flight at once: a load under a divergent branch
  // would make the compiler wait for it at the branch's join.
  auto load_rows = [&](uint4 (&x)[RPI][CH], uint4 (&y)[RPI][CH], int it) {
#pragma unroll
    for (int u = 0; u < RPI; ++u) {
      const int i = qb * R + wave + 4 * (it * RPI + u);
      const int last = d.causal ? min(s_valid - V, i / V * V) : s_valid - V;
#pragma unroll
      for (int t = 0; t < CH; ++t) {
        const int jc = min((lc + 64 * t) * V, last);
        x[u][t] = *reinterpret_cast<const uint4*>(src + int64_t(i) * S + jc);
        if (BWD) y[u][t] = *reinterpret_cast<const uint4*>(src2 + int64_t(i) * S + jc);
      }
    }
  };
  // live keys of the chunk starting at j0 in query row i: a prefix of it
  auto n_live = [&](int j0, int i) {
    return d.causal ? min(V, max(0, i - j0 + 1)) : (j0 < S ? V : 0);
  };
  // chunk t of row i is live in every lane (inside s_valid and, under the
  // mask, at or before the diagonal): a wave-uniform test that skips the
  // per-element selects
  auto full = [&](int t, int i) {
    const int hi = 64 * (t + 1) * V;
    return hi <= s_valid && (!d.causal || hi - 1 <= i);
  };
  const int n_it = R / (4 * RPI);
  // With PF an iteration's stores (the output chunks and, for R = 128, the
  // row checksum pairs) are issued in the next iteration, after its wait:
  // the compiler's wait for loaded data also drains every store in flight,
  // so stores issued just before a wait would stall it.
  uint4 pb[RPI][CH];
  float2 prc[RPI][CH];
  const bool rc_late = PF && PERM && CHK && R == 128 && d.row_chk != nullptr;
  auto flush = [&](int it) {
#pragma unroll
    for (int u = 0; u < RPI; ++u) {
      const int i = qb * R + wave + 4 * (it * RPI + u);
#pragma unroll
      for (int t = 0; t < CH; ++t) {
        if (64 * t * V >= s_valid) continue;
        const int j0 = (lc + 64 * t) * V;
        if (j0 < s_valid) *reinterpret_cast<uint4*>(dst + int64_t(i) * S + j0) = pb[u][t];
        const int k0 = 64 * t * V + 128 * (lane >> 4);
        if (rc_late && (lane & 15) == 0 && k0 < s_valid)
          *reinterpret_cast<float2*>(d.row_chk + ((int64_t(z) * S + i) * nq + k0 / 128) * 2) =
              prc[u][t];
      }
    }
  };
  auto process_rows = [&](uint4 (&xr)[RPI][CH], uint4 (&yr)[RPI][CH], int it) {
    // keys a chunk holds past s_valid, or past the diagonal, are the
    // masked tail of its live prefix (n_live), which is all that the
    // arithmetic below masks
    float xs[RPI][CH][V], ys[RPI][CH][V];
#pragma unroll
    for (int u = 0; u < RPI; ++u)
#pragma unroll
      for (int t = 0; t < CH; ++t) {
        Vec<T>::unpack(xr[u][t], xs[u][t]);
        if (BWD) Vec<T>::unpack(yr[u][t], ys[u][t]);
      }
    if constexpr (PF) {
      // The load registers are free once unpacked: the next iteration's
      // loads go out now and run during this iteration's arithmetic. The
      // empty statements pin that order (the wait for this iteration's
      // data, which also drains the stores still in flight, comes first;
      // a load hoisted above it would be waited for at once).
#pragma unroll
      for (int u = 0; u < RPI; ++u)
#pragma unroll
        for (int t = 0; t < CH; ++t)
#pragma unroll
          for (int e = 0; e < V; ++e) {
            asm volatile("" : "+v"(xs[u][t][e]));
            if (BWD) asm volatile("" : "+v"(ys[u][t][e]));
          }
      asm volatile("" ::: "memory");
      if (it + 1 < n_it) load_rows(xr, yr, it + 1);
      if (it > 0) flush(it - 1);
    }
#pragma unroll
    for (int u = 0; u < RPI; ++u) {
      const int rl = wave + 4 * (it * RPI + u);
      const int i = qb * R + rl;
      float* const rc_row = d.row_chk + (int64_t(z) * S + i) * nq * 2;  // [S / R][2] of row i
      float (&x)[CH][V] = xs[u];
      float (&y)[CH][V] = ys[u];
      // chunk t holds data only if 64 t V < s_valid (a wave-uniform test)
      if (!BWD) {
        // AP = softmax(scale * AS) over live keys, in base 2
        const float sc = d.scale * l2e;
        float mx = -INFINITY;
#pragma unroll
        for (int t = 0; t < CH; ++t) {
          if (64 * t * V >= s_valid) continue;
          if (!full(t, i)) {
            const int nl = n_live((lc + 64 * t) * V, i);
#pragma unroll
            for (int e = 0; e < V; ++e) x[t][e] = e < nl ? x[t][e] : -INFINITY;
          }
#pragma unroll
          for (int e = 0; e < V; ++e) mx = fmaxf(mx, x[t][e]);
        }
        mx = wave_max(mx);
        const float mo = -mx * sc;
        float sum = 0.f;
#pragma unroll
        for (int t = 0; t < CH; ++t) {
          if (64 * t * V >= s_valid) continue;
#pragma unroll
          for (int e = 0; e < V; ++e) {
            x[t][e] = __builtin_amdgcn_exp2f(fmaf(x[t][e], sc, mo));  // masked: exp2(-inf) = 0
            sum += x[t][e];
          }
        }
        const float inv = 1.f / wave_sum(sum);
#pragma unroll
        for (int t = 0; t < CH; ++t)
#pragma unroll
          for (int e = 0; e < V; ++e) x[t][e] *= inv;
      } else {
        // dAS = scale * AP * (dAP - D), D = sum_j AP_j dAP_j over live keys;
        // masked keys are zeroed in both operands (so that they add nothing
        // to D whatever they hold) and in the result (exactly zero even
        // when D is not finite)
        float dot = 0.f;
#pragma unroll
        for (int t = 0; t < CH; ++t) {
          if (64 * t * V >= s_valid) continue;
          if (!full(t, i)) {  // wave-uniform: full chunks skip the selects
            const int nl = n_live((lc + 64 * t) * V, i);
#pragma unroll
            for (int e = 0; e < V; ++e) {
              x[t][e] = e < nl ? x[t][e] : 0.f;
              y[t][e] = e < nl ? y[t][e] : 0.f;
            }
          }
#pragma unroll
          for (int e = 0; e < V; ++e) dot = fmaf(x[t][e], y[t][e], dot);
        }
        dot = wave_sum(dot);
        const float nsd = -d.scale * dot;
#pragma unroll
        for (int t = 0; t < CH; ++t) {
          if (64 * t * V >= s_valid) continue;
          if (full(t, i)) {
#pragma unroll
            for (int e = 0; e < V; ++e) x[t][e] *= fmaf(y[t][e], d.scale, nsd);
          } else {
            const int nl = n_live((lc + 64 * t) * V, i);
#pragma unroll
            for (int e = 0; e < V; ++e) {
              const float v = x[t][e] * fmaf(y[t][e], d.scale, nsd);
              x[t][e] = e < nl ? v : 0.f;
            }
          }
        }
      }
      // round, store, accumulate column checksums, emit row checksums per
      // key block (weights 1..R inside the block: base + e + 1)
      const float wr = float(rl + 1);
#pragma unroll
      for (int t = 0; t < CH; ++t) {
        if (64 * t * V >= s_valid) continue;
        const int j0 = (lc + 64 * t) * V;
        uint4 bits;
        round_chunk(x[t], bits);
        float r1 = 0.f, rw = 0.f;
        if constexpr (PF) pb[u][t] = bits;
        if (j0 < s_valid) {
          if constexpr (!PF) *reinterpret_cast<uint4*>(dst + int64_t(i) * S + j0) = bits;
          if constexpr (CHK) {
#pragma unroll
            for (int e = 0; e < V; ++e) {
              c1[t][e] += x[t][e];
              c2[t][e] = fmaf(wr, x[t][e], c2[t][e]);
              if constexpr (!PERM) {
                r1 += x[t][e];
                rw = fmaf(float(e), x[t][e], rw);
              }
            }
          }
        }
        if constexpr (PERM) {
          if (CHK && d.row_chk != nullptr) {
            // D[m][0] = sum of quarter m, D[m][1] = its in-quarter weighted
            // sum; lane (n, g) holds rows 4g..4g+3 of column n, lane n = 1's
            // column reaches lane n = 0 by a pair swap
            const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
            const floatx4 dq =
                __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, bits), bsum, zero, 0, 0, 0);
            floatx4 dw;
#pragma unroll
            for (int r = 0; r < 4; ++r) dw[r] = dpp_mov<DPP_XOR1>(dq[r]);
            // lane group g = lane / 16 (lane 16 g holds its sums) covers
            // keys k0 .. k0 + 127: one key block of R = 128, or 128 / R
            // whole blocks, whose checksum pairs are contiguous in the row's
            // [S / R][2] record
            const int k0 = 64 * t * V + 128 * (lane >> 4);
            if (rc_late) {
              prc[u][t] = make_float2((dq[0] + dq[1]) + (dq[2] + dq[3]),
                                      ((dw[0] + dq[0]) + (dw[1] + 33.f * dq[1])) +
                                          ((dw[2] + 65.f * dq[2]) + (dw[3] + 97.f * dq[3])));
            } else if ((lane & 15) == 0 && k0 < s_valid) {
              float q1[4], q2[4];  // per 32-key quarter: sum, weighted sum
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                q1[r] = dq[r];
                q2[r] = dw[r] + float(((32 * r) & (R - 1)) + 1) * dq[r];
              }
              float* rc = rc_row + (k0 / R) * 2;
              if (R == 128) {
                *reinterpret_cast<float2*>(rc) =
                    make_float2((q1[0] + q1[1]) + (q1[2] + q1[3]), (q2[0] + q2[1]) + (q2[2] + q2[3]));
              } else if (R == 64) {
                *reinterpret_cast<float2*>(rc) = make_float2(q1[0] + q1[1], q2[0] + q2[1]);
                if (k0 + 64 < s_valid)
                  *reinterpret_cast<float2*>(rc + 2) = make_float2(q1[2] + q1[3], q2[2] + q2[3]);
              } else {  // R == 32
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  if (k0 + 32 * r < s_valid)
                    *reinterpret_cast<float2*>(rc + 2 * r) = make_float2(q1[r], q2[r]);
              }
            }
          }
        } else if (CHK && d.row_chk != nullptr) {
          float r2 = fmaf(float((j0 & (R - 1)) + 1), r1, rw);
          kb_sums(r1, r2, lanes_per_kb);
          if ((lane % lanes_per_kb) == 0 && j0 < s_valid) {
            float* rc = d.row_chk + ((int64_t(z) * S + i) * nq + j0 / R) * 2;
            rc[0] = r1;
            rc[1] = r2;
          }
        }
      }
    }
  };

  uint4 xa[RPI][CH], ya[RPI][CH];
  if constexpr (PF) load_rows(xa, ya, 0);
  for (int it = 0; it < n_it; ++it) {
    if constexpr (!PF) load_rows(xa, ya, it);
    process_rows(xa, ya, it);
  }
  if constexpr (PF) flush(n_it - 1);

  // combine the four waves' column checksums in a fixed order: each wave's
  // partials go to a slab of its own, then every thread sums the four
  // slabs for its columns
  if (CHK && d.col_chk != nullptr) {
    float* p1 = colacc;          // [4][S]
    float* p2 = colacc + 4 * S;  // [4][S]
#pragma unroll
    for (int t = 0; t < CH; ++t)
#pragma unroll
      for (int e = 0; e < V; ++e) {
        const int j = (lc + 64 * t) * V + e;
        if (j < s_valid) {
          p1[wave * S + j] = c1[t][e];
          p2[wave * S + j] = c2[t][e];
        }
      }
    __syncthreads();
    float* cc = d.col_chk + (int64_t(z) * nq + qb) * 2 * S;
    for (int j = tid; j < s_valid; j += NT) {
      cc[j] = ((p1[j] + p1[S + j]) + p1[2 * S + j]) + p1[3 * S + j];
      cc[S + j] = ((p2[j] + p2[S + j]) + p2[2 * S + j]) + p2[3 * S + j];
    }
  }
}

// CUs per XCD of the current device (8 XCDs), read once per device
int xcd_cus() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    v = cus / 8 > 0 ? cus / 8 : -1;
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return v > 0 ? v : 0;
}

template <bool BWD>
hipError_t launch_sm(const SoftmaxDesc& desc, int dtype, hipStream_t s) {
  SoftmaxDesc d = desc;
  d.xcd_cus = xcd_cus();
  const int V = dtype == ABFT_FP32 ? 4 : 8;
  // key blocks: a power of two, whole 16-byte lane chunks, at most one
  // 128-key lane group (bf16: whole 32-key MFMA quarters)
  if ((d.R & (d.R - 1)) != 0 || d.R > 128 || d.R < (dtype == ABFT_FP32 ? 16 : 32))
    return hipErrorInvalidValue;
  const int ch = (d.S + 64 * V - 1) / (64 * V);
  dim3 grid(unsigned((d.S / d.R) * d.B * d.nh));
  const size_t lds = size_t(d.S) * 8 * sizeof(float);
  const bool chk = d.col_chk != nullptr || d.row_chk != nullptr;
#define SM_CASE(TT, CHV)                                                                      \
  if (ch <= CHV) {                                                                            \
    auto k = chk ? softmax_kernel<TT, CHV, BWD, (CHV == 1 ? 2 : 1), (CHV <= 2), true>         \
                 : softmax_kernel<TT, CHV, BWD, (CHV == 1 ? 2 : 1), (CHV <= 2), false>;       \
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
