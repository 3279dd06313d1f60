// Direct-to-LDS operand loads and their fragment reads (bf16), shared by
// the GEMM and the fused attention kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "abft_device.hpp"

namespace abft {
namespace {

// ---- direct-to-LDS operand path (bf16) ------------------------------------
// A stage's operand tile goes from global memory straight into LDS
// (global_load_lds_dwordx4: lane p of a wave instruction writes bytes
// [16p, 16p + 16) of a 1-KB LDS run, from any 16-byte global address), so
// no registers hold it and several stages can be in flight. The LDS images
// are unpadded and XOR-swizzled at 16-byte granularity so that the MFMA
// fragment reads do not conflict on banks:
//  - K-major tile [ROWS][64]: chunk c of row r lives at chunk c ^ (r & 7)
//    (the 8 rows a b128 read serves together hit 8 different chunks);
//  - MN-major tile [64][ROWS] (one row per k): chunk c of k-row k lives at
//    chunk c ^ 2 (k & 3) (the 4 k-rows a transposing read serves together
//    hit 4 different chunk pairs).
// MN-major fragments are read with ds_read_b64_tr_b16: in each group of 16
// lanes, lane s supplies the 4 elements at (k0 + s/4, m0 + 4 (s%4)), and
// lane i receives element i%4 of lanes i/4, i/4 + 4, i/4 + 8, i/4 + 12,
// i.e. (k0 + v, m0 + i) for v = 0..3: the k-contiguous MFMA operand.
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) short4_t lds_short4;

// ds_read_b64_tr_b16 as inline assembly. Through the compiler's intrinsic,
// the read first waits for every outstanding direct-to-LDS load of the
// wave (vmcnt 0), which serialises the next stage's loads with the
// compute on the current one (the stage being read is already complete:
// the loop's own wait and barrier see to that). The compiler does not see
// this LDS access, so its result is read only after lds_wait_all() and
// through tr_join(), which redefines it behind the wait.
__device__ __forceinline__ short4_t ds_read_tr16(const void* p) {
  short4_t r;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"((const lds_short4*)p));
  return r;
}
// Waits for every outstanding LDS access of the wave.
__device__ __forceinline__ void lds_wait_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// Waits until at most the last two LDS accesses of the wave are outstanding
// (LDS accesses complete in order, so every earlier one is done).
__device__ __forceinline__ void lds_wait_but2() { asm volatile("s_waitcnt lgkmcnt(2)" ::: "memory"); }
// The two transposed halves of an MN-major fragment (k rows 0..3 and 4..7
// of the lane's 8), as read, before the wait.
struct TrPair {
  short4_t lo, hi;
};
__device__ __forceinline__ TrPair tr_pair(const void* p0, const void* p1) {
  return TrPair{ds_read_tr16(p0), ds_read_tr16(p1)};
}
// The same through the compiler's intrinsic (it waits for the loads into
// LDS itself; fewer registers where the assembly form spills).
__device__ __forceinline__ TrPair tr_pair_intrinsic(const void* p0, const void* p1) {
  return TrPair{__builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4*)p0),
                __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4*)p1)};
}
// After lds_wait_all(): the fragment. The empty statements redefine both
// halves behind the wait, so no copy of them is taken before it.
__device__ __forceinline__ bf16x8 tr_join(TrPair& t) {
  asm volatile("" : "+v"(t.lo));
  asm volatile("" : "+v"(t.hi));
  typedef short short8_t __attribute__((ext_vector_type(8)));
  const short8_t v = {t.lo[0], t.lo[1], t.lo[2], t.lo[3], t.hi[0], t.hi[1], t.hi[2], t.hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

template <bool KMAJ, int ROWS, int NT = 256>
struct Direct {
  static constexpr int BK = 64;
  static constexpr int BYTES = ROWS * BK * 2;
  static constexpr int PER_WAVE = BYTES / 1024 / (NT / 64);  // 1-KB instructions per wave
  static_assert(BYTES % (1024 * (NT / 64)) == 0, "tile must split into whole wave runs");

  // rows past nrows read a clamped (valid) row: their results are never stored
  __device__ static __forceinline__ void issue(const bf16_t* base, int64_t ld, int row0, int nrows,
                                               int k0, char* st, int wave, int lane) {
#pragma unroll
    for (int j = 0; j < PER_WAVE; ++j) {
      const int i = wave * PER_WAVE + j;
      const bf16_t* src;
      if constexpr (KMAJ) {
        const int row = i * 8 + (lane >> 3);
        const int c = (lane & 7) ^ (row & 7);
        src = base + int64_t(min(row0 + row, nrows - 1)) * ld + k0 + c * 8;
      } else {
        constexpr int CPR = ROWS / 8;       // 16-byte chunks per k-row
        constexpr int KR = 64 / CPR;        // k-rows per 1-KB run
        const int kr = i * KR + lane / CPR;
        const int c = (lane % CPR) ^ (2 * (kr & 3));
        src = base + int64_t(k0 + kr) * ld + min(row0 + c * 8, nrows - 8);
      }
      __builtin_amdgcn_global_load_lds(src, (lds_void*)(st + i * 1024), 16, 0, 0);
    }
  }

  // MFMA 16x16x32 operand fragment: rows rb + (lane & 15), k = kk + 8 (lane >> 4) + 0..7
  // (K-major image: a plain LDS read)
  __device__ static __forceinline__ bf16x8 frag(const char* st, int rb, int kk, int lane) {
    static_assert(KMAJ, "MN-major fragments: frag_tr, then lds_wait_all and tr_join");
    const int row = rb + (lane & 15);
    const int c = (kk >> 3) + (lane >> 4);
    return *reinterpret_cast<const bf16x8*>(st + row * 128 + ((c ^ (row & 7)) << 4));
  }
  // the same fragment from an MN-major image, as two transposing reads
  __device__ static __forceinline__ TrPair frag_tr(const char* st, int rb, int kk, int lane) {
    static_assert(!KMAJ, "K-major fragments: frag");
    const int s = lane & 15;
    const int k = kk + 8 * (lane >> 4) + (s >> 2);
    const int m = rb + 4 * (s & 3);
    const int c = m >> 3, off = (m & 7) * 2;
    const char* p0 = st + k * (ROWS * 2) + ((c ^ (2 * (k & 3))) << 4) + off;
    const char* p1 = st + (k + 4) * (ROWS * 2) + ((c ^ (2 * ((k + 4) & 3))) << 4) + off;
    return tr_pair(p0, p1);
  }
};

// s_waitcnt that waits for the vector-memory counter only (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14, expcnt and lgkmcnt left at their maxima)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

}  // namespace
}  // namespace abft
