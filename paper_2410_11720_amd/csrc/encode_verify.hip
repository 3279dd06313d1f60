// Checksum encoder (paper Sec. 4.6 "Encoding") and the standalone EEC-ABFT
// verifier (Sec. 4.2, 4.3) behind encode_checksums / verify_and_correct.
//
// Encoder: one workgroup owns an Rb-row block of one batch matrix and a
// slab of columns; a thread owns 16-byte column chunks (coalesced row
// reads) and accumulates the column checksums of its chunk in registers;
// row checksums of each Cb-column block are reduced across the lanes that
// hold the block. The whole operand is read exactly once.
//
// Verifier: one workgroup per (batch, Rb-row block); one thread per vector
// (the paper's Fig. 4 thread-per-vector mapping); a clean block costs one
// coalesced read. Corrections use the checksums only (DELTA or
// RECONSTRUCT), since no operands are at hand.
#include "abft_internal.hpp"
#include "abft_device.hpp"

namespace abft {
namespace {

constexpr int NT = 256;

template <class T, int V>
__device__ __forceinline__ void load_vec(const T* p, float* out) {
  if constexpr (V == 8 && sizeof(T) == 2) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      out[2 * q] = __uint_as_float(w[q] << 16);
      out[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
    }
  } else if constexpr (V == 4 && sizeof(T) == 4) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
  } else {
#pragma unroll
    for (int e = 0; e < V; ++e) out[e] = Storage<T>::load(p[e]);
  }
}

// grid: (ceil(cols / (CPS*V)), rows/Rb, batch). A workgroup owns an
// Rb-row block and a slab of CPS 16-byte chunks per row; thread (c, g)
// holds chunk c of rows g, g+RG, ... (RG = 256/CPS row groups), all of its
// loads in flight together. Column checksums are combined over the row
// groups in LDS in a fixed order; row checksums of each Cb-column block
// are reduced across the Cb/V lanes that hold it (consecutive lanes share
// a row), which needs Cb/V a power of two dividing CPS.
template <class T, int V, int CPS>
__device__ __forceinline__ void encode_block(const T* A, int64_t rows, int64_t cols, int64_t ld,
                                             int64_t bstride, int Rb, int Cb, float* col_chk,
                                             float* row_chk, int64_t bx, int64_t rb, int64_t b,
                                             int64_t ldcc, uint16_t* col_img, int64_t ldci,
                                             uint16_t* row_img, int64_t ldri) {
  constexpr int RG = NT / CPS, W = CPS * V;
  __shared__ float part[RG][W][2];
  // the transposed row-checksum image of this workgroup's blocks, staged
  // so that it leaves in 16-byte row pieces: [4][block of the slab][row]
  constexpr int RIMG = 1024;
  __shared__ __align__(16) uint16_t rimg[4][RIMG];
  const int c = threadIdx.x % CPS, g = threadIdx.x / CPS;
  const int64_t c0 = bx * W + c * V;
  const bool live = c0 < cols;
  const T* base = A + b * bstride + rb * Rb * ld;
  const int lanes = Cb / V;
  const float wb = float((c0 % Cb) + 1);  // weight of the chunk's first column in its block
  const int nbs = W / Cb;                 // column blocks of the slab (W is a multiple of Cb)
  const bool stage_ri = row_img != nullptr && nbs * Rb <= RIMG && Rb % 8 == 0 && ldri % 8 == 0 &&
                        reinterpret_cast<uintptr_t>(row_img) % 16 == 0;
  float c1[V], c2[V];
#pragma unroll
  for (int e = 0; e < V; ++e) c1[e] = c2[e] = 0.f;
  for (int r0 = g; r0 < Rb; r0 += 4 * RG) {
    // unconditional loads from clamped addresses, zeroed afterwards (a
    // load under a divergent branch is waited for at the join)
    float x[4][V];
    const int64_t cc = live ? c0 : cols - V;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = min(r0 + RG * u, Rb - 1);
      load_vec<T, V>(base + r * ld + cc, x[u]);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const bool ok = live && r0 + RG * u < Rb;
#pragma unroll
      for (int e = 0; e < V; ++e) x[u][e] = ok ? x[u][e] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = r0 + RG * u;
      float s1 = 0.f, sw = 0.f;
#pragma unroll
      for (int e = 0; e < V; ++e) {
        c1[e] += x[u][e];
        c2[e] = fmaf(float(r + 1), x[u][e], c2[e]);
        s1 += x[u][e];
        sw = fmaf(float(e), x[u][e], sw);
      }
      if (row_chk != nullptr && r0 + RG * u - g < Rb) {  // uniform: the wave's rows exist
        float s2 = fmaf(wb, s1, sw);
        s1 = group_sum_n(s1, lanes);
        s2 = group_sum_n(s2, lanes);
        if (live && r < Rb && (c0 % Cb) == 0) {
          float* rc = row_chk + ((b * rows + rb * Rb + r) * (cols / Cb) + c0 / Cb) * 2;
          rc[0] = s1;
          rc[1] = s2;
          if (row_img != nullptr) {  // the transposed bf16 image: hi and lo rows
            const bf16_t h1 = f2bf(s1), h2 = f2bf(s2);
            const bf16_t v[4] = {h1, f2bf(s1 - bf2f(h1)), h2, f2bf(s2 - bf2f(h2))};
            if (stage_ri) {
              const int e = int((c0 % W) / Cb) * Rb + r;
#pragma unroll
              for (int q = 0; q < 4; ++q) rimg[q][e] = v[q];
            } else {
              uint16_t* ip = row_img + (4 * (c0 / Cb)) * ldri + b * rows + rb * Rb + r;
#pragma unroll
              for (int q = 0; q < 4; ++q) ip[q * ldri] = v[q];
            }
          }
        }
      }
    }
  }
  if (stage_ri) {  // every row of the block is staged: 16-byte pieces out
    __syncthreads();
    const int pieces = Rb / 8;
    for (int u = threadIdx.x; u < 4 * nbs * pieces; u += NT) {
      const int q = u / (nbs * pieces), bs = (u / pieces) % nbs, pc = u % pieces;
      const int64_t blk = bx * W / Cb + bs;
      if (blk * Cb < cols)
        *reinterpret_cast<uint4*>(row_img + (4 * blk + q) * ldri + b * rows + rb * Rb + pc * 8) =
            *reinterpret_cast<const uint4*>(&rimg[q][bs * Rb + pc * 8]);
    }
  }
  if (col_chk != nullptr) {
#pragma unroll
    for (int e = 0; e < V; ++e) {
      part[g][c * V + e][0] = c1[e];
      part[g][c * V + e][1] = c2[e];
    }
    __syncthreads();
    const int col = threadIdx.x % W, which = threadIdx.x / W;  // 2W <= NT threads
    if (threadIdx.x < 2 * W && bx * W + col < cols) {
      float acc = 0.f;
      for (int q = 0; q < RG; ++q) acc += part[q][col][which];
      col_chk[((b * (rows / Rb) + rb) * 2 + which) * ldcc + bx * W + col] = acc;
      if (col_img != nullptr) {  // the bf16 image: hi and lo rows of this checksum
        const bf16_t hi = f2bf(acc), lo = f2bf(acc - bf2f(hi));
        uint16_t* ip = col_img + ((b * (rows / Rb) + rb) * 4 + 2 * which) * ldci + bx * W + col;
        ip[0] = hi;
        ip[ldci] = lo;
      }
    }
  }
}

template <class T, int V, int CPS>
__global__ __launch_bounds__(NT) void encode_kernel(const T* A, int64_t rows, int64_t cols,
                                                    int64_t ld, int64_t bstride, int Rb, int Cb,
                                                    float* col_chk, float* row_chk) {
  encode_block<T, V, CPS>(A, rows, cols, ld, bstride, Rb, Cb, col_chk, row_chk, blockIdx.x,
                          blockIdx.y, blockIdx.z, cols, nullptr, 0, nullptr, 0);
}

__device__ __forceinline__ void clear_counters(abft_report* rep) {
  rep->n_events = 0;
  rep->n_corrected = 0;
  rep->n_uncorrectable = 0;
  rep->overflow = 0;
}

// Up to two encodes in one launch (a one-dimensional grid, the first job's
// workgroups first), and optionally the report's counters cleared by the
// first workgroup: nothing in an encode records events, and the kernels
// after it in the stream start once it has finished.
struct EncJob {
  const void* A;
  int64_t rows, cols, ld, bs;
  int Rb, Cb;
  float* col_chk;
  float* row_chk;
  unsigned gx, gy, nblk;  // workgroups: gx column slabs x gy row blocks x batch
  int64_t ldcc;           // elements between column-checksum rows
  uint16_t* col_img;      // optional bf16 image of the column checksums
  int64_t ldci;
  uint16_t* row_img;      // optional transposed bf16 image of the row checksums
  int64_t ldri;
};

template <class T, int V, int CPS>
__device__ __forceinline__ void encode_job(const EncJob& j, unsigned id) {
  const unsigned bx = id % j.gx, by = (id / j.gx) % j.gy, bz = id / (j.gx * j.gy);
  encode_block<T, V, CPS>(static_cast<const T*>(j.A), j.rows, j.cols, j.ld, j.bs, j.Rb, j.Cb,
                          j.col_chk, j.row_chk, bx, by, bz, j.ldcc, j.col_img, j.ldci,
                          j.row_img, j.ldri);
}

template <class T, int V, int CPS>
__global__ __launch_bounds__(NT) void encode_jobs_kernel(EncJob j0, EncJob j1, EncJob j2,
                                                         abft_report* reset) {
  const unsigned id = blockIdx.x;
  if (reset != nullptr && id == 0 && threadIdx.x == 0) clear_counters(reset);
  if (id < j0.nblk)
    encode_job<T, V, CPS>(j0, id);
  else if (id < j0.nblk + j1.nblk)
    encode_job<T, V, CPS>(j1, id - j0.nblk);
  else
    encode_job<T, V, CPS>(j2, id - j0.nblk - j1.nblk);
}

// Row checksums for block widths the lane-group reduction cannot cover:
// one thread per (row, block), sequential sums.
template <class T>
__global__ __launch_bounds__(NT) void row_chk_kernel(const T* A, int64_t batch, int64_t rows,
                                                     int64_t cols, int64_t ld, int64_t bstride,
                                                     int Cb, float* row_chk) {
  const int64_t nb = cols / Cb;
  const int64_t idx = int64_t(blockIdx.x) * NT + threadIdx.x;
  if (idx >= batch * rows * nb) return;
  const int64_t cb = idx % nb, row = (idx / nb) % rows, b = idx / (nb * rows);
  const T* p = A + b * bstride + row * ld + cb * Cb;
  float s1 = 0.f, s2 = 0.f;
  for (int k = 0; k < Cb; ++k) {
    const float x = Storage<T>::load(p[k]);
    s1 += x;
    s2 += float(k + 1) * x;
  }
  row_chk[idx * 2] = s1;
  row_chk[idx * 2 + 1] = s2;
}

template <class T>
hipError_t encode_t(const T* A, int64_t batch, int64_t rows, int64_t cols, int64_t ld,
                    int64_t bs, int Rb, int Cb, float* col_chk, float* row_chk, hipStream_t s) {
  constexpr int VV = 16 / sizeof(T);
  const bool aligned = (reinterpret_cast<uintptr_t>(A) % 16 == 0) && (ld % VV == 0) &&
                       (cols % VV == 0) && (bs % VV == 0);
  // slab of CPS chunks: 8, or 16 when a row-checksum block needs it
  int cps = 8;
  bool rows_inline = row_chk == nullptr;
  if (aligned && row_chk != nullptr && Cb % VV == 0) {
    const int l = Cb / VV;
    if ((l & (l - 1)) == 0 && l <= 16) {
      rows_inline = true;
      cps = l > 8 ? 16 : 8;
    }
  }
  float* rc_inline = (row_chk != nullptr && rows_inline) ? row_chk : nullptr;
  if (aligned && (col_chk != nullptr || rc_inline != nullptr)) {
    const int W = cps * VV;
    dim3 grid(unsigned((cols + W - 1) / W), unsigned(rows / Rb), unsigned(batch));
    if (cps == 8)
      hipLaunchKernelGGL((encode_kernel<T, VV, 8>), grid, dim3(NT), 0, s, A, rows, cols, ld, bs,
                         Rb, Cb, col_chk, rc_inline);
    else
      hipLaunchKernelGGL((encode_kernel<T, VV, 16>), grid, dim3(NT), 0, s, A, rows, cols, ld, bs,
                         Rb, Cb, col_chk, rc_inline);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  } else if (col_chk != nullptr) {  // unaligned operand: scalar chunks (V = 1)
    dim3 grid(unsigned((cols + 8 * 1 - 1) / 8), unsigned(rows / Rb), unsigned(batch));
    hipLaunchKernelGGL((encode_kernel<T, 1, 8>), grid, dim3(NT), 0, s, A, rows, cols, ld, bs, Rb,
                       Cb, col_chk, nullptr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    rows_inline = row_chk == nullptr;
  }
  if (row_chk != nullptr && !(aligned && rows_inline)) {
    const int64_t n = batch * rows * (cols / Cb);
    hipLaunchKernelGGL((row_chk_kernel<T>), dim3(unsigned((n + NT - 1) / NT)), dim3(NT), 0, s, A,
                       batch, rows, cols, ld, bs, Cb, row_chk);
    return hipGetLastError();
  }
  return hipSuccess;
}

// ---- standalone verify-and-correct ---------------------------------------

// Global-memory reads in the verifier must observe corrections made by
// other threads of the workgroup: they go through the device-coherent
// level after a workgroup barrier with a device-scope fence.
__device__ __forceinline__ void wg_sync_global() {
  __threadfence();
  __syncthreads();
  __threadfence();
}

template <class T>
__global__ __launch_bounds__(NT) void verify_kernel(T* C, int64_t rows, int64_t cols, int64_t ld,
                                                    int64_t bstride, int Rb, int Cb,
                                                    float* col_chk, float* row_chk, float tn,
                                                    float tc, float e_rel, int op_tag,
                                                    abft_report* rep) {
  extern __shared__ __align__(16) char smem[];
  int* rowcnt = reinterpret_cast<int*>(smem);          // [Rb][cols/Cb]
  const int64_t b = blockIdx.y, rb = blockIdx.x;
  const int64_t nrb = row_chk ? cols / Cb : 0;
  int* colcnt = rowcnt + Rb * nrb;                     // [cols]
  T* M = C + b * bstride + rb * Rb * ld;
  float* cc = col_chk + ((b * (rows / Rb) + rb) * 2) * cols;
  float* rc = row_chk ? row_chk + (b * rows + rb * Rb) * nrb * 2 : nullptr;
  const int tid = threadIdx.x;
  for (int64_t e = tid; e < Rb * nrb + (row_chk ? cols : 0); e += NT) rowcnt[e] = 0;

  // quick clean check: any flagged vector?
  bool my = false;
  for (int64_t n = tid; n < cols; n += NT)
    my |= vec_flagged<T>(M + n, int(ld), Rb, cc[n], e_rel);
  if (row_chk)
    for (int64_t u = tid; u < Rb * nrb; u += NT)
      my |= vec_flagged<T>(M + (u / nrb) * ld + (u % nrb) * Cb, 1, Cb, rc[u * 2], e_rel);
  if (!__syncthreads_or(my)) return;

  auto fix = [&](T* vec, int stride, int n, int idx, float c1, float d1, int row, int col) {
    const float old = Storage<T>::load(vec[idx * stride]);
    int action;
    const float val = fix_by_checksum<T>(vec, stride, n, idx, c1, d1, tc, &action);
    vec[idx * stride] = Storage<T>::store(val);
    record_event(rep, op_tag, int(b), 0, row, col, classify(old, tn), action, old);
  };
  // 1. column pass
  for (int64_t n = tid; n < cols; n += NT) {
    T* vec = M + n;
    const EecResult r = eec_locate<T>(vec, int(ld), Rb, cc[n], cc[cols + n], e_rel, tn);
    if (r.status == EEC_LOCATED) {
      fix(vec, int(ld), Rb, r.index, cc[n], r.d1, int(rb * Rb + r.index), int(n));
      if (row_chk) atomicAdd(&rowcnt[r.index * nrb + n / Cb], 1);
    }
  }
  wg_sync_global();
  if (row_chk) {
    // 2a. refresh row checksums of 1R-corrected row vectors
    for (int64_t u = tid; u < Rb * nrb; u += NT)
      if (rowcnt[u] >= 2)
        vec_checksums<T>(M + (u / nrb) * ld + (u % nrb) * Cb, 1, Cb, &rc[u * 2], &rc[u * 2 + 1]);
    wg_sync_global();
    // 2b. row pass
    for (int64_t u = tid; u < Rb * nrb; u += NT) {
      const int64_t row = u / nrb, cb = u % nrb;
      T* vec = M + row * ld + cb * Cb;
      const EecResult r = eec_locate<T>(vec, 1, Cb, rc[u * 2], rc[u * 2 + 1], e_rel, tn);
      if (r.status == EEC_LOCATED) {
        fix(vec, 1, Cb, r.index, rc[u * 2], r.d1, int(rb * Rb + row), int(cb * Cb + r.index));
        atomicAdd(&colcnt[cb * Cb + r.index], 1);
      }
    }
    wg_sync_global();
    // 2c. refresh column checksums of 1C-corrected column vectors
    for (int64_t n = tid; n < cols; n += NT)
      if (colcnt[n] >= 2) vec_checksums<T>(M + n, int(ld), Rb, &cc[n], &cc[cols + n]);
    wg_sync_global();
  }
  // 3. final check
  for (int64_t n = tid; n < cols; n += NT)
    if (vec_flagged<T>(M + n, int(ld), Rb, cc[n], e_rel))
      record_event(rep, op_tag, int(b), 0, int(rb * Rb), int(n), ABFT_KIND_NONE,
                   ABFT_ACT_UNCORRECTABLE, 0.f);
  if (row_chk)
    for (int64_t u = tid; u < Rb * nrb; u += NT)
      if (vec_flagged<T>(M + (u / nrb) * ld + (u % nrb) * Cb, 1, Cb, rc[u * 2], e_rel))
        record_event(rep, op_tag, int(b), 0, int(rb * Rb + u / nrb), int((u % nrb) * Cb),
                     ABFT_KIND_NONE, ABFT_ACT_UNCORRECTABLE, 0.f);
}

__global__ void report_reset_kernel(abft_report* rep, int capacity, int set_capacity) {
  if (threadIdx.x == 0) {
    clear_counters(rep);
    if (set_capacity) {
      rep->capacity = capacity;
      rep->reserved[0] = rep->reserved[1] = rep->reserved[2] = 0;
    }
  }
}

}  // namespace

hipError_t launch_encode(const void* A, int dtype, int64_t batch, int64_t rows, int64_t cols,
                         int64_t ld, int64_t batch_stride, int Rb, int Cb, float* col_chk,
                         float* row_chk, hipStream_t s) {
  if (batch == 0 || rows == 0 || cols == 0) return hipSuccess;
  if (dtype == ABFT_FP32)
    return encode_t<float>(static_cast<const float*>(A), batch, rows, cols, ld, batch_stride, Rb,
                           Cb, col_chk, row_chk, s);
  return encode_t<bf16_t>(static_cast<const bf16_t*>(A), batch, rows, cols, ld, batch_stride, Rb,
                          Cb, col_chk, row_chk, s);
}

namespace {
// The bf16 image of dense column checksums ([nrow][cols] fp32, two rows per
// block) for the separate-launch form: image rows 2r (hi) and 2r + 1 (lo).
__global__ __launch_bounds__(NT) void chk_image_kernel(const float* chk, int64_t nrow,
                                                       int64_t cols, uint16_t* img, int64_t ldci) {
  const int64_t i = int64_t(blockIdx.x) * NT + threadIdx.x;
  if (i >= nrow * cols) return;
  const int64_t r = i / cols, c = i % cols;
  const float v = chk[i];
  const bf16_t hi = f2bf(v), lo = f2bf(v - bf2f(hi));
  img[(2 * r) * ldci + c] = hi;
  img[(2 * r + 1) * ldci + c] = lo;
}

// The transposed bf16 image of row checksums ([nrow][nblk][2] fp32) for the
// separate-launch form: image rows 4 blk + (0 hi c1, 1 lo c1, 2 hi c2, 3 lo
// c2), column = the operand row.
__global__ __launch_bounds__(NT) void rowchk_image_kernel(const float* chk, int64_t nrow,
                                                          int64_t nblk, uint16_t* img,
                                                          int64_t ldri) {
  const int64_t i = int64_t(blockIdx.x) * NT + threadIdx.x;
  if (i >= nrow * nblk) return;
  const int64_t r = i / nblk, blk = i % nblk;
#pragma unroll
  for (int w = 0; w < 2; ++w) {
    const float v = chk[i * 2 + w];
    const bf16_t hi = f2bf(v);
    img[(4 * blk + 2 * w) * ldri + r] = hi;
    img[(4 * blk + 2 * w + 1) * ldri + r] = f2bf(v - bf2f(hi));
  }
}

// The single-launch form applies when every job takes the vector path with
// its row checksums inline and the same slab width.
template <class T>
bool job_of(const EncodeJob& e, EncJob& j, int& cps) {
  constexpr int VV = 16 / sizeof(T);
  const bool aligned = (reinterpret_cast<uintptr_t>(e.A) % 16 == 0) && (e.ld % VV == 0) &&
                       (e.cols % VV == 0) && (e.batch_stride % VV == 0);
  if (!aligned || (e.col_chk == nullptr && e.row_chk == nullptr)) return false;
  cps = 8;
  if (e.row_chk != nullptr) {
    if (e.Cb % VV != 0) return false;
    const int l = e.Cb / VV;
    if ((l & (l - 1)) != 0 || l > 16) return false;
    cps = l > 8 ? 16 : 8;
  }
  const int64_t W = int64_t(cps) * VV;
  const int64_t gx = (e.cols + W - 1) / W, gy = e.rows / e.Rb, n = gx * gy * e.batch;
  if (n <= 0 || n > (int64_t(1) << 30)) return false;
  j = EncJob{e.A, e.rows, e.cols, e.ld, e.batch_stride, e.Rb, e.Cb, e.col_chk, e.row_chk,
             unsigned(gx), unsigned(gy), unsigned(n), e.ldcc > 0 ? e.ldcc : e.cols,
             e.col_img, e.ldci, e.row_img, e.ldri};
  return true;
}

template <class T>
hipError_t encode_jobs_t(const EncodeJob* jobs, int n, abft_report* reset, hipStream_t s) {
  EncJob j[3] = {};
  int cps[3] = {8, 8, 8};
  bool one = n >= 1 && n <= 3;
  for (int i = 0; one && i < n; ++i) one = job_of<T>(jobs[i], j[i], cps[i]);
  for (int i = 1; one && i < n; ++i) one = cps[i] == cps[0];
  if (!one) {  // separate launches
    if (reset != nullptr) {
      hipError_t e = launch_report_reset(reset, 0, false, s);
      if (e != hipSuccess) return e;
    }
    for (int i = 0; i < n; ++i) {
      const EncodeJob& e = jobs[i];
      // the separate kernels write dense column checksums only
      if (e.col_chk != nullptr && e.ldcc > 0 && e.ldcc != e.cols) return hipErrorInvalidValue;
      hipError_t r = launch_encode(e.A, sizeof(T) == 4 ? ABFT_FP32 : ABFT_BF16, e.batch, e.rows,
                                   e.cols, e.ld, e.batch_stride, e.Rb, e.Cb, e.col_chk,
                                   e.row_chk, s);
      if (r != hipSuccess) return r;
      if (e.col_img != nullptr && e.col_chk != nullptr) {
        const int64_t nrow = e.batch * (e.rows / e.Rb) * 2, nel = nrow * e.cols;
        const unsigned nb = unsigned((nel + NT - 1) / NT);
        hipLaunchKernelGGL(chk_image_kernel, dim3(nb), dim3(NT), 0, s, e.col_chk, nrow, e.cols,
                           e.col_img, e.ldci);
        if ((r = hipGetLastError()) != hipSuccess) return r;
      }
      if (e.row_img != nullptr && e.row_chk != nullptr) {
        const int64_t nrow = e.batch * e.rows, nblk = e.cols / e.Cb;
        const unsigned nb = unsigned((nrow * nblk + NT - 1) / NT);
        hipLaunchKernelGGL(rowchk_image_kernel, dim3(nb), dim3(NT), 0, s, e.row_chk, nrow, nblk,
                           e.row_img, e.ldri);
        if ((r = hipGetLastError()) != hipSuccess) return r;
      }
    }
    return hipSuccess;
  }
  constexpr int VV = 16 / sizeof(T);
  unsigned total = 0;
  for (int i = 0; i < n; ++i) total += j[i].nblk;   // unused jobs have nblk 0
  if (cps[0] == 8)
    hipLaunchKernelGGL((encode_jobs_kernel<T, VV, 8>), dim3(total), dim3(NT), 0, s, j[0], j[1],
                       j[2], reset);
  else
    hipLaunchKernelGGL((encode_jobs_kernel<T, VV, 16>), dim3(total), dim3(NT), 0, s, j[0], j[1],
                       j[2], reset);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_encode_jobs(const EncodeJob* jobs, int n, int dtype, abft_report* reset,
                              hipStream_t s) {
  // empty operands encode nothing
  EncodeJob live[3];
  int m = 0;
  for (int i = 0; i < n; ++i)
    if (jobs[i].batch > 0 && jobs[i].rows > 0 && jobs[i].cols > 0) {
      if (m == 3) return hipErrorInvalidValue;
      live[m++] = jobs[i];
    }
  if (m == 0) return reset != nullptr ? launch_report_reset(reset, 0, false, s) : hipSuccess;
  if (dtype == ABFT_FP32) return encode_jobs_t<float>(live, m, reset, s);
  return encode_jobs_t<bf16_t>(live, m, reset, s);
}

hipError_t launch_verify(void* C, int dtype, int64_t batch, int64_t rows, int64_t cols,
                         int64_t ld, int64_t batch_stride, int Rb, int Cb, float* col_chk,
                         float* row_chk, float tn, float tc, float e_rel, int op_tag,
                         abft_report* report, hipStream_t s) {
  if (batch == 0 || rows == 0 || cols == 0) return hipSuccess;
  const int64_t nrb = row_chk ? cols / Cb : 0;
  const size_t lds = size_t(Rb * nrb + (row_chk ? cols : 0)) * sizeof(int);
  dim3 grid(rows / Rb, batch);
  if (dtype == ABFT_FP32) {
    auto k = verify_kernel<float>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k, grid, dim3(NT), lds, s, static_cast<float*>(C), rows, cols, ld,
                       batch_stride, Rb, Cb, col_chk, row_chk, tn, tc, e_rel, op_tag, report);
  } else {
    auto k = verify_kernel<bf16_t>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k, grid, dim3(NT), lds, s, static_cast<bf16_t*>(C), rows, cols, ld,
                       batch_stride, Rb, Cb, col_chk, row_chk, tn, tc, e_rel, op_tag, report);
  }
  return hipGetLastError();
}

hipError_t launch_report_reset(abft_report* report, int capacity, bool set_capacity,
                               hipStream_t s) {
  hipLaunchKernelGGL(report_reset_kernel, dim3(1), dim3(64), 0, s, report, capacity,
                     set_capacity ? 1 : 0);
  return hipGetLastError();
}

}  // namespace abft
