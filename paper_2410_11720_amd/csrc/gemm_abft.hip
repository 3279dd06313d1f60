// Protected GEMM for gfx950: C = A B on MFMA 16x16x32 bf16 (or 16x16x4
// f32), with the ABFT checksums of paper Sec. 2.3 carried as extra MFMA
// tiles (the "packed operand" update of Sec. 4.6): the column checksums
// A^c of the tile's row blocks form a 16-row strip that is multiplied by
// the same B fragments (C^c = A^c B), and, for two-sided outputs, the row
// checksums B^r form a 16-column strip multiplied by the same A fragments
// (C^r = A B^r). fp32 checksums enter a bf16 MFMA as a hi + lo bf16 pair,
// so the propagated checksum keeps ~16 significant bits.
//
// The epilogue rounds the tile to storage and stages it in LDS, applies
// injected faults, and compares recomputed against propagated checksums,
// one thread per checksum vector (detection, Sec. 2.3). A flagged tile is
// corrected in LDS: EEC-ABFT on every column vector (Sec. 4.2), and for
// two-sided outputs the row pass with the checksum refresh of Sec. 4.3,
// then a final check; located elements are recomputed from A and B (or
// corrected from the checksums when the operands are not trusted) and
// every action is appended to the device report. The tile then leaves LDS
// in 16-byte coalesced stores.
#include <algorithm>

#include "abft_internal.hpp"
#include "abft_device.hpp"
#include "direct_lds.hpp"

namespace abft {

namespace {

constexpr int NT = 256;  // threads per workgroup: 4 waves as 2 (M) x 2 (N)

// The kernel's descriptor (argument `slot` of the kernel: the descriptors
// are its first arguments), reached through an opaque copy of the
// kernel-argument segment address: fields read through it are loaded where
// they are used instead of being held in scalar registers from the
// kernel's start.
__device__ __forceinline__ const GemmDesc& desc_reload(int slot) {
#if defined(__HIP_DEVICE_COMPILE__)
  // the copy stays in the constant address space, so the fields are read
  // with scalar loads
  auto gp = __builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(gp));
  return *((const GemmDesc*)gp + slot);
#else
  return *static_cast<const GemmDesc*>(nullptr);  // the host pass emits no device code
#endif
}

template <class T> struct Mfma;
template <> struct Mfma<bf16_t> {
  static constexpr int BK = 64;    // k per LDS stage (128 bytes per row)
  static constexpr int KI = 32;    // k per instruction
  static constexpr int PAD = 8;    // 16 bytes of padding per LDS row
  typedef bf16x8 frag;
  __device__ static frag load(const bf16_t* p) { return *reinterpret_cast<const frag*>(p); }
  __device__ static floatx4 mma(frag a, frag b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  static constexpr int BK = 32;
  static constexpr int KI = 4;
  static constexpr int PAD = 4;
  typedef float frag;
  __device__ static frag load(const float* p) { return *p; }
  __device__ static floatx4 mma(frag a, frag b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// Element offset of operand element (row, k) of an M x K (or N x K) operand.
template <bool KMAJ>
__device__ __forceinline__ int64_t op_off(int64_t row, int64_t k, int64_t ld) {
  return KMAJ ? row * ld + k : k * ld + row;
}

// Global -> registers -> LDS loader of one ROWS x BK operand tile; the LDS
// image is k-contiguous per row ([ROWS][BK + PAD]) whatever the global
// layout. A K-major source is copied in 16-byte chunks; an MN-major source
// is read as VEC x VEC blocks (VEC rows of k, VEC consecutive rows each),
// one block per thread, and transposed in registers.
template <class T, bool KMAJ, int ROWS>
struct TileLoader {
  static constexpr int BK = Mfma<T>::BK;
  static constexpr int LDK = BK + Mfma<T>::PAD;
  static constexpr int VEC = 16 / sizeof(T);
  static constexpr int CHUNKS = ROWS * BK / VEC;            // 16-byte chunks per tile
  static constexpr int NRB = ROWS / VEC, NBLK = NRB * (BK / VEC);
  static constexpr int PER = KMAJ ? (CHUNKS + NT - 1) / NT : ((NBLK + NT - 1) / NT) * VEC;
  uint4 reg[PER];

  __device__ void load(const T* base, int64_t ld, int row0, int nrows, int k0, int kend,
                       int tid) {
    // interior tiles (the common case) skip the per-chunk bounds tests
    const bool full = row0 + ROWS <= nrows && k0 + BK <= kend;
    if constexpr (KMAJ) {
      if (full && CHUNKS % NT == 0) {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
          const int c = tid + p * NT;
          const int r = c / (BK / VEC), kc = (c % (BK / VEC)) * VEC;
          reg[p] = *reinterpret_cast<const uint4*>(base + op_off<true>(row0 + r, k0 + kc, ld));
        }
        return;
      }
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        const int c = tid + p * NT;
        const int r = c / (BK / VEC), kc = (c % (BK / VEC)) * VEC;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (c < CHUNKS && row0 + r < nrows && k0 + kc < kend)
          v = *reinterpret_cast<const uint4*>(base + op_off<true>(row0 + r, k0 + kc, ld));
        reg[p] = v;
      }
    } else {
#pragma unroll
      for (int p = 0; p < PER / VEC; ++p) {
        const int blk = tid + p * NT;
        const int rb = blk % NRB, kb = blk / NRB;
#pragma unroll
        for (int s = 0; s < VEC; ++s) {
          uint4 v = make_uint4(0, 0, 0, 0);
          if (blk < NBLK && row0 + rb * VEC < nrows && k0 + kb * VEC + s < kend)
            v = *reinterpret_cast<const uint4*>(
                base + op_off<false>(row0 + rb * VEC, k0 + kb * VEC + s, ld));
          reg[p * VEC + s] = v;
        }
      }
    }
  }

  __device__ void store(T* lds, int tid) {
    if constexpr (KMAJ) {
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        const int c = tid + p * NT;
        if (c < CHUNKS) {
          const int r = c / (BK / VEC), kc = (c % (BK / VEC)) * VEC;
          *reinterpret_cast<uint4*>(lds + r * LDK + kc) = reg[p];
        }
      }
    } else {
#pragma unroll
      for (int p = 0; p < PER / VEC; ++p) {
        const int blk = tid + p * NT;
        if (blk >= NBLK) continue;
        const int rb = blk % NRB, kb = blk / NRB;
        uint32_t in[VEC][4];
#pragma unroll
        for (int s = 0; s < VEC; ++s) {
          in[s][0] = reg[p * VEC + s].x;
          in[s][1] = reg[p * VEC + s].y;
          in[s][2] = reg[p * VEC + s].z;
          in[s][3] = reg[p * VEC + s].w;
        }
#pragma unroll
        for (int e = 0; e < VEC; ++e) {  // output row rb*VEC + e, k = kb*VEC + [0, VEC)
          uint4 out;
          if constexpr (sizeof(T) == 2) {
            const int dw = e >> 1;
            uint32_t o[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const uint32_t a = in[2 * q][dw], b = in[2 * q + 1][dw];
              o[q] = (e & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
            }
            out = make_uint4(o[0], o[1], o[2], o[3]);
          } else {
            out = make_uint4(in[0][e], in[1][e], in[2][e], in[3][e]);
          }
          *reinterpret_cast<uint4*>(lds + (rb * VEC + e) * LDK + kb * VEC) = out;
        }
      }
    }
  }
};

// Checksum strip loader: NC fp32 checksum rows (laid out like the operand)
// for the tile, stored as NC fp32 rows, or for bf16 operands as a hi and a
// lo row each, interleaved (row 2r hi, 2r + 1 lo): the strip rows of
// checksum block b are 4b (hi c1), 4b + 1 (lo c1), 4b + 2 (hi c2), 4b + 3
// (lo c2).
template <class T, bool KMAJ>
struct StripLoader {
  static constexpr int BK = Mfma<T>::BK;
  static constexpr int LDK = BK + Mfma<T>::PAD;
  // fp32 source rows a strip can hold: 16 strip rows, two (hi, lo) per
  // source row for bf16 operands
  static constexpr int NR = sizeof(T) == 2 ? 8 : 16;
  static constexpr int PER = (NR * BK + NT - 1) / NT;
  float reg[PER];

  // Element e of the strip: consecutive threads walk the contiguous
  // direction of the source (k for a K-major strip, the checksum row for an
  // MN-major one), so the loads coalesce.
  __device__ static void rk(int e, int& r, int& k) {
    if (KMAJ) { r = e / BK; k = e % BK; }
    else { r = e % NR; k = e / NR; }
  }
  // rows r0 + r exist only for r < nvalid (the last tile may be ragged)
  __device__ void load(const float* base, int64_t ld, int r0, int nvalid, int k0, int kend,
                       int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int e = tid + p * NT;
      int r, k;
      rk(e, r, k);
      float v = 0.f;
      if (r < nvalid && k0 + k < kend) v = base[op_off<KMAJ>(r0 + r, k0 + k, ld)];
      reg[p] = v;
    }
  }
  __device__ void store(T* lds, int nc, int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int e = tid + p * NT;
      int r, k;
      rk(e, r, k);
      if (r < nc) {
        if constexpr (sizeof(T) == 2) {
          const bf16_t hi = f2bf(reg[p]);
          const bf16_t lo = f2bf(reg[p] - bf2f(hi));
          lds[(2 * r) * LDK + k] = hi;
          lds[(2 * r + 1) * LDK + k] = lo;
        } else {
          lds[r * LDK + k] = reg[p];
        }
      }
    }
  }
};

struct EvCoord {
  int op, b, h, row, col;
};
__device__ __forceinline__ EvCoord map_coord(const CoordMap& mp, int z, int m, int n) {
  EvCoord c;
  c.op = mp.op_base + n / mp.op_span;
  const int nn = n % mp.op_span;
  if (mp.nb1 > 0) {
    c.b = z / mp.nb1;
    c.h = z % mp.nb1;
    c.row = m;
    c.col = nn;
  } else {
    c.b = mp.rows_per_b ? m / mp.rows_per_b : 0;
    c.row = mp.rows_per_b ? m % mp.rows_per_b : m;
    c.h = mp.head_cols ? nn / mp.head_cols : 0;
    c.col = mp.head_cols ? nn % mp.head_cols : nn;
  }
  return c;
}

// Inverse of map_coord for a fault; returns false if op is not produced here.
__device__ __forceinline__ bool fault_target(const CoordMap& mp, int N, const abft_fault& f,
                                             int* z, int* m, int* n) {
  const int nops = (N + mp.op_span - 1) / mp.op_span;
  if (f.op < mp.op_base || f.op >= mp.op_base + nops) return false;
  const int nbase = (f.op - mp.op_base) * mp.op_span;
  if (mp.nb1 > 0) {
    *z = f.b * mp.nb1 + f.h;
    *m = f.row;
    *n = nbase + f.col;
  } else {
    *z = 0;
    *m = mp.rows_per_b ? f.b * mp.rows_per_b + f.row : f.row;
    *n = nbase + (mp.head_cols ? f.h * mp.head_cols : 0) + f.col;
  }
  return true;
}

template <class T, class TC, bool AK, bool BKM>
__device__ float recompute_elem(const GemmDesc& g, const T* A, const T* B, int m, int n, int k_lo,
                                int k_hi) {
  float s = 0.f;
#pragma unroll 8
  for (int k = k_lo; k < k_hi; ++k)
    s = fmaf(Storage<T>::load(A[op_off<AK>(m, k, g.lda)]),
             Storage<T>::load(B[op_off<BKM>(n, k, g.ldb)]), s);
  return s;
}

// Work item of a workgroup. The grid is one-dimensional and the hardware
// deals consecutive workgroup ids round-robin to the 8 XCDs (each with its
// own L2), so the decode decides both the balance and the L2 locality:
//  - batched GEMMs (one per batch x head) put the head index fastest, so
//    each XCD gets whole heads (their operands stay in its L2) and every
//    XCD sees the same mix of tile costs;
//  - causally trimmed K ranges run the most expensive tile rows first;
//  - a causal score GEMM (whole tiles above the diagonal skipped)
//    enumerates only the lower-triangle tiles;
//  - unbatched GEMMs give each XCD one contiguous range of tiles, walked
//    in bands of GM tile rows, column by column (GM = 1024 / BM), so that
//    the tiles an XCD runs at once share about 1024 rows of A and 1024
//    columns of B in its L2; split-K slices keep their K range together.
struct TileIdx {
  int mt, nt, bh, ks;
};

__host__ __device__ inline bool tri_tiles(const GemmDesc& g, int bm, int bn) {
  return g.causal == 1 && bm == bn && g.M == g.N;
}

template <int BM, int BN>
__device__ __forceinline__ TileIdx tile_of(const GemmDesc& g, int lin, int total) {
  const int ntm = (g.M + BM - 1) / BM, ntn = (g.N + BN - 1) / BN;
  const int nb = g.nb0 * g.nb1;
  TileIdx t;
  int r;
  if (nb == 1) {
    const int q = total / 8, rem = total % 8;
    const int x = lin % 8, j = lin / 8;
    const int v = x * q + min(x, rem) + j;
    const int per = tri_tiles(g, BM, BN) ? ntm * (ntm + 1) / 2 : ntm * ntn;
    t.bh = 0;
    t.ks = v / per;
    r = v % per;
  } else {
    t.bh = lin % nb;
    t.ks = 0;
    r = lin / nb;
  }
  if (nb == 1 && g.causal == 0) {
    constexpr int GM = BM >= 1024 ? 1 : 1024 / BM;
    const int band = r / (GM * ntn), idx = r % (GM * ntn);
    const int rows_in_band = min(GM, ntm - band * GM);
    t.mt = band * GM + idx % rows_in_band;
    t.nt = idx / rows_in_band;
  } else if (tri_tiles(g, BM, BN)) {  // r -> (mt, nt) with nt <= mt
    int mt = int((sqrtf(8.f * r + 1.f) - 1.f) * 0.5f);
    while ((mt + 1) * (mt + 2) / 2 <= r) ++mt;
    while (mt * (mt + 1) / 2 > r) --mt;
    t.mt = mt;
    t.nt = r - mt * (mt + 1) / 2;
  } else if (g.causal == 2) {  // K range grows with the tile row
    t.mt = ntm - 1 - r / ntn;
    t.nt = r % ntn;
  } else {
    t.mt = r / ntn;
    t.nt = r % ntn;
  }
  return t;
}

// WLC: wave-local column check. The four waves split the tile's columns
// (each holds all BM rows of BN / 4 columns), so every column checksum
// block lies inside one wave: the wave sums, decides and stores its part
// without a workgroup barrier (outputs checked on the column side only).
// Otherwise the waves form a 2 x 2 grid.
template <class T, class TC, bool AK, bool BKM, int BM, int BN, bool PROT, int NSTAGE,
          bool WLC = false>
struct Gemm {
  static constexpr int BK = Mfma<T>::BK;
  static constexpr int KI = Mfma<T>::KI;
  static constexpr int LDK = BK + Mfma<T>::PAD;
  static constexpr int WGN = WLC ? 4 : 2, WGM = 4 / WGN;  // wave grid
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int IM = WM / 16, JN = WN / 16;
  // strip blocks per wave: column strips of the wave's own columns (WLC)
  // or split between the two waves sharing them; row strips split between
  // the waves sharing the rows
  static constexpr int JS = WLC ? JN : JN / 2, IS = IM / WGN;
  static_assert(WLC ? (IM >= 4 && JN >= 1) : (IM >= 2 && JN >= 2), "tile too small");
  static constexpr int FRAG = KI / 4;  // operand elements per lane
  // bf16 operands and bf16 output: detection sums on the matrix cores
  static constexpr bool MSUM = PROT && sizeof(T) == 2 && sizeof(TC) == 2;

  // LDS map of the main loop: per stage the A and B tiles, then the
  // checksum strips the GEMM carries (column strip, row strip), so a GEMM
  // with one strip keeps two workgroups per CU.
  static constexpr int A_ELEMS = BM * LDK, B_ELEMS = BN * LDK, S_ELEMS = 16 * LDK;
  __host__ __device__ static constexpr int stage_elems(bool cc, bool cr) {
    return A_ELEMS + B_ELEMS + (PROT ? ((cc ? S_ELEMS : 0) + (cr ? S_ELEMS : 0)) : 0);
  }
  // the register path uses at most two stages
  static constexpr int RSTAGES = NSTAGE >= 2 ? 2 : 1;
  __host__ __device__ static constexpr size_t main_bytes(bool cc, bool cr) {
    return size_t(RSTAGES) * stage_elems(cc, cr) * sizeof(T);
  }
  // direct path: unpadded swizzled operand images, the strips as above
  static constexpr int DA_BYTES = BM * 64 * 2, DB_BYTES = BN * 64 * 2;
  __host__ __device__ static constexpr int d_stage_bytes(bool cc, bool cr) {
    return DA_BYTES + DB_BYTES +
           (PROT ? ((cc ? S_ELEMS : 0) + (cr ? S_ELEMS : 0)) * int(sizeof(T)) : 0);
  }
  __host__ __device__ static constexpr size_t d_main_bytes(bool cc, bool cr) {
    return size_t(NSTAGE) * d_stage_bytes(cc, cr);
  }
  // LDS map of the epilogue (overlays the operand stages once the K loop is
  // done): the rounded tile [BM][LDT], then one region that first holds
  // the strip results ([16][BN] column strip, [BM][16] row strip), then,
  // once those are read, the combined propagated checksums and the
  // detection's segment sums, and last the correction counters and queue
  // (in the segment sums' place). Sized so that a 128 x 128 bf16 tile keeps
  // three workgroups per CU.
  static constexpr int MINB = sizeof(T) == 2 ? 32 : 16;  // smallest checksum block
  static constexpr int TPAD = 16 / sizeof(TC);
  static constexpr int LDT = BN + TPAD;
  static constexpr size_t TILE_BYTES = size_t(BM) * LDT * sizeof(TC);
  // bf16 operands with fp32 output are the weight gradients, checked on
  // the column side only: no row strip, no row checksums (the launch
  // refuses them), so that an unsplit checked tile keeps two workgroups
  // per CU
  static constexpr bool COLS_ONLY = sizeof(T) == 2 && sizeof(TC) == 4;
  static constexpr size_t STRIPS = 16 * BN + (COLS_ONLY ? 0 : 16 * BM);
  // checksum pairs ([BM/MINB][BN][2], [BM][BN/MINB][2]); the segment sums
  // (sum, magnitude) have the same shapes
  static constexpr size_t CCV = (BM / MINB) * BN * 2, RCV = COLS_ONLY ? 0 : BM * (BN / MINB) * 2;
  static constexpr size_t CNT = BM * (BN / MINB) + (BM / MINB) * BN;
  // recompute queue of the correction passes: count, QMAX x (row, col,
  // observed value), and one partial sum per wave
  static constexpr int QMAX = 32;
  static constexpr size_t QUE = 1 + 3 * QMAX + NT / 64;
  static constexpr size_t WORK = CCV + RCV > CNT + QUE ? CCV + RCV : CNT + QUE;
  static constexpr size_t EREG = STRIPS > CCV + RCV + WORK ? STRIPS : CCV + RCV + WORK;
  static constexpr size_t EPI_BYTES = TILE_BYTES + (PROT ? EREG * 4 : 0);
  __host__ __device__ static constexpr size_t lds_bytes(bool cc, bool cr) {
    return main_bytes(cc, cr) > EPI_BYTES ? main_bytes(cc, cr) : EPI_BYTES;
  }

  // DIR selects the direct-to-LDS operand path (bf16 only) at compile time,
  // so each kernel carries the registers and code of one path only.
  template <bool DIR>
  // lin, total: the workgroup's index among this GEMM's workgroups and
  // their count (a launch of two GEMMs deals each its own range; the first
  // range is a multiple of 8 long, so both keep the dealing to the XCDs);
  // slot: the descriptor's argument slot
  __device__ static __forceinline__ void run(const GemmDesc& g, char* smem, int lin, int total,
                                             int slot) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    const TileIdx ti = tile_of<BM, BN>(g, lin, total);
    const int m0 = ti.mt * BM, n0 = ti.nt * BN;
    const int z = ti.bh, kslice = ti.ks;
    const int b0 = z / g.nb1, b1 = z % g.nb1;
    if (g.causal == 1 && n0 > m0 + BM - 1) return;  // whole tile above the diagonal

    int k_lo = 0, k_hi = g.K;
    if (g.causal == 2) k_hi = min(g.K, m0 + BM);
    if (g.causal == 3) k_lo = min(g.K, m0);
    const bool split = g.splitk > 1;
    if (split) {  // K slice of this workgroup, a multiple of BK
      const int kc = ((g.K + g.splitk - 1) / g.splitk + BK - 1) / BK * BK;
      k_lo = min(g.K, kslice * kc);
      k_hi = min(g.K, k_lo + kc);
    }

    const T* A = static_cast<const T*>(g.A) + b0 * g.sA0 + b1 * g.sA1;
    const T* B = static_cast<const T*>(g.B) + b0 * g.sB0 + b1 * g.sB1;
    TC* C = static_cast<TC*>(g.C) + b0 * g.sC0 + b1 * g.sC1 + int64_t(kslice) * g.sCk;

    // whether an injected fault (test-only) lands in this tile: the list is
    // read here, and only such tiles take the injection step of the
    // epilogue (with its barriers)
    bool wf = false;
    if (g.n_faults > 0 && !split) {
      for (int f = 0; f < g.n_faults; ++f) {
        const abft_fault ft = g.faults[f];
        int fz, fm, fn;
        wf |= fault_target(g.map, g.N, ft, &fz, &fm, &fn) && fz == z && fm >= m0 &&
              fm < m0 + BM && fn >= n0 && fn < n0 + BN;
      }
    }

    const bool cc = PROT && g.Ac != nullptr;
    const bool cr = PROT && g.Br != nullptr && n0 >= g.cr_n_begin;
    // checksum block sizes are powers of two (the launch checks): shifts
    const int lg_rm = __builtin_ctz(g.Rm), lg_rn = __builtin_ctz(g.Rn);
    const int nc = cc ? 2 * (BM >> lg_rm) : 0;       // checksum rows of this tile
    const int nq = cr ? 2 * (BN >> lg_rn) : 0;       // checksum cols of this tile
    const int rc0 = 2 * (m0 >> lg_rm);
    const int qc0 = cr ? 2 * ((n0 - g.cr_n_begin) >> lg_rn) : 0;
    const int nc_valid = cc ? min(nc, 2 * (g.M >> lg_rm) - rc0) : 0;
    const int nq_valid = cr ? min(nq, 2 * ((g.N - g.cr_n_begin) >> lg_rn) - qc0) : 0;
    const float* Ac = cc ? g.Ac + b0 * g.sAc0 + b1 * g.sAc1 : nullptr;
    const float* Br = cr ? g.Br + b0 * g.sBr0 + b1 * g.sBr1 : nullptr;

    T* lds = reinterpret_cast<T*>(smem);
    // stage stride and row-strip offset follow the strips this GEMM carries
    const bool g_cc = PROT && g.Ac != nullptr, g_cr = PROT && g.Br != nullptr;
    const int STAGE = stage_elems(g_cc, g_cr);
    const int r_off = g_cc ? S_ELEMS : 0;
    TileLoader<T, AK, BM> la;
    TileLoader<T, BKM, BN> lb;
    StripLoader<T, AK> ls;
    StripLoader<T, BKM> lr;

    floatx4 acc[IM][JN];
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int j = 0; j < JN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    // strip results: the two waves sharing columns (rows) split them
    floatx4 accs[JS], accr[IS];
#pragma unroll
    for (int j = 0; j < JS; ++j) accs[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < IS; ++i) accr[i] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int nk = k_hi > k_lo ? (k_hi - k_lo + BK - 1) / BK : 0;
    const int fr = lane & 15, fk = (lane >> 4) * FRAG;
    // the checksum strips' fragments of one KI-wide k step, read with the
    // tile's fragments so that one wait covers them all (a GEMM without a
    // column strip reads the stage's first rows instead: a valid address,
    // the value unused)
    using Frag = typename Mfma<T>::frag;
    // the column strip copied from its bf16 image (direct path): 2 nc rows
    // of 64 elements, unpadded; fragment rows past them repeat the rows
    // (their MFMA result rows are not read)
    // (the one-stage tile, held to three workgroups per CU, keeps the strip
    // reads after the tile's MFMAs and per-lane selects: fewer live
    // registers; it has no images)
    constexpr bool EARLY = NSTAGE >= 2;
    bool img = false, imgr = false;
    if constexpr (DIR && EARLY) {
      img = cc && g.Aci != nullptr && nc_valid > 0;
      imgr = cr && g.Bri != nullptr && nq_valid > 0;
    }
    const int soff = img ? (fr & (2 * nc - 1)) * BK + fk : fr * LDK + fk;
    const int roff = imgr ? (fr & (2 * nq - 1)) * BK + fk : fr * LDK + fk;
    auto strip_frags = [&](const T* st0, const T* sS, const T* sR, int kk, Frag& sf, Frag& rf) {
      if (PROT && EARLY) {
        sf = Mfma<T>::load((cc ? sS + soff : st0 + fr * LDK + fk) + kk);
        if (cr) rf = Mfma<T>::load(sR + roff + kk);
      }
    };
    // the waves' positions in the wave grid as scalars: the strip blocks a
    // wave multiplies are chosen by uniform branches, so every fragment
    // index stays a compile-time constant (a runtime index would send the
    // arrays to scratch) and no per-lane selects are spent on them
    const int wmu = __builtin_amdgcn_readfirstlane(wm), wnu = __builtin_amdgcn_readfirstlane(wn);
    // the MFMAs of one KI-wide k step: the tile, then the checksum strips
    auto mma_kk = [&](const Frag (&af)[IM], const Frag (&bfr)[JN], const Frag& sf,
                      const Frag& rf, const T* sS, const T* sR, int kk) {
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int j = 0; j < JN; ++j) acc[i][j] = Mfma<T>::mma(af[i], bfr[j], acc[i][j]);
      if (PROT && !EARLY) {
        if (cc) {
          const auto sfl = Mfma<T>::load(sS + fr * LDK + kk + fk);
#pragma unroll
          for (int j = 0; j < JS; ++j) {
            const auto bsel = (WLC || wm == 0) ? bfr[j] : bfr[WLC ? j : JS + j];
            accs[j] = Mfma<T>::mma(sfl, bsel, accs[j]);
          }
        }
        if (cr) {
          const auto rfl = Mfma<T>::load(sR + fr * LDK + kk + fk);
#pragma unroll
          for (int i = 0; i < IS; ++i) {
            auto asel = af[i];
#pragma unroll
            for (int w = 1; w < WGN; ++w) asel = wn == w ? af[IS * w + i] : asel;
            accr[i] = Mfma<T>::mma(rfl, asel, accr[i]);
          }
        }
      }
      if (PROT && EARLY) {
        if (cc) {
          if (WLC || wmu == 0) {
#pragma unroll
            for (int j = 0; j < JS; ++j) accs[j] = Mfma<T>::mma(sf, bfr[j], accs[j]);
          } else {
#pragma unroll
            for (int j = 0; j < JS; ++j) accs[j] = Mfma<T>::mma(sf, bfr[WLC ? j : JS + j], accs[j]);
          }
        }
        if (cr) {
#pragma unroll
          for (int w = 0; w < WGN; ++w)
            if (wnu == w) {
#pragma unroll
              for (int i = 0; i < IS; ++i) accr[i] = Mfma<T>::mma(rf, af[IS * w + i], accr[i]);
            }
        }
      }
    };

    if constexpr (DIR) {
      static_assert(sizeof(T) == 2, "the direct path is for bf16 operands");
      {
        // Direct path: NSTAGE LDS stages, operand loads issued NSTAGE - 1
        // stages ahead; the strips go through registers one stage ahead,
        // issued before the operand loads of the same iteration so that
        // waiting for them never waits for later operand stages.
        using DA = Direct<AK, BM>;
        using DB = Direct<BKM, BN>;
        constexpr int NDIR = DA::PER_WAVE + DB::PER_WAVE;  // vector-memory ops per wave and stage
        const int DST = d_stage_bytes(g_cc, g_cr);
        const bf16_t* Ab = reinterpret_cast<const bf16_t*>(A);
        const bf16_t* Bb = reinterpret_cast<const bf16_t*>(B);
        auto slot = [&](int kt) { return smem + (kt % NSTAGE) * DST; };
        auto issue_dir = [&](int kt) {
          char* st = slot(kt);
          DA::issue(Ab, g.lda, m0, g.M, k_lo + kt * BK, st, wave, lane);
          DB::issue(Bb, g.ldb, n0, g.N, k_lo + kt * BK, st + DA_BYTES, wave, lane);
        };
        auto issue_strip = [&](int kt) {
          const int kn = k_lo + kt * BK;
          if (cc && !img) ls.load(Ac, g.ldac, rc0, nc_valid, kn, k_hi, tid);
          if (cr && !imgr) lr.load(Br, g.ldbr, qc0, nq_valid, kn, k_hi, tid);
        };
        auto commit_strip = [&](int kt) {
          T* st = reinterpret_cast<T*>(slot(kt) + DA_BYTES + DB_BYTES);
          if (cc && !img) ls.store(st, nc, tid);
          if (cr && !imgr) lr.store(st + r_off, nq, tid);
        };
        // the strips from their images: the column strip's rows go to
        // waves 0.., the row strip's to the waves after them; a wave copies
        // eight image rows (eight 16-byte chunks each) into the stage's strip
        // region; rows past the tile's valid ones read its last valid row
        const int wc = img ? (2 * nc + 7) / 8 : 0;
        auto issue_img = [&](int kt) {
          if (img && wave < wc) {
            const int r = min(wave * 8 + (lane >> 3), 2 * nc_valid - 1);
            const uint16_t* src =
                g.Aci + int64_t(2 * rc0 + r) * g.ldaci + k_lo + kt * BK + (lane & 7) * 8;
            __builtin_amdgcn_global_load_lds(
                src, (lds_void*)(slot(kt) + DA_BYTES + DB_BYTES + wave * 1024), 16, 0, 0);
          }
          if (imgr && wave >= wc && (wave - wc) * 8 < 2 * nq) {
            const int w = wave - wc;
            const int r = min(w * 8 + (lane >> 3), 2 * nq_valid - 1);
            const uint16_t* src =
                g.Bri + int64_t(2 * qc0 + r) * g.ldbri + k_lo + kt * BK + (lane & 7) * 8;
            __builtin_amdgcn_global_load_lds(
                src,
                (lds_void*)(slot(kt) + DA_BYTES + DB_BYTES + r_off * int(sizeof(T)) + w * 1024),
                16, 0, 0);
          }
        };
        auto compute_d = [&](const char* st) {
          const T* sS = reinterpret_cast<const T*>(st + DA_BYTES + DB_BYTES);
          const T* sR = sS + r_off;
#pragma unroll
          for (int kk = 0; kk < BK; kk += KI) {
            typename Mfma<T>::frag af[IM], bfr[JN];
            // MN-major images are read with transposing reads that are
            // waited for together
            TrPair ap[AK ? 1 : IM], bp[BKM ? 1 : JN];
#pragma unroll
            for (int i = 0; i < IM; ++i) {
              if constexpr (AK) af[i] = DA::frag(st, wm * WM + i * 16, kk, lane);
              else ap[i] = DA::frag_tr(st, wm * WM + i * 16, kk, lane);
            }
#pragma unroll
            for (int j = 0; j < JN; ++j) {
              if constexpr (BKM) bfr[j] = DB::frag(st + DA_BYTES, wn * WN + j * 16, kk, lane);
              else bp[j] = DB::frag_tr(st + DA_BYTES, wn * WN + j * 16, kk, lane);
            }
            Frag sf, rf;
            strip_frags(reinterpret_cast<const T*>(st), sS, sR, kk, sf, rf);
            if constexpr (!AK || !BKM) {
              lds_wait_all();
              if constexpr (!AK) {
#pragma unroll
                for (int i = 0; i < IM; ++i) af[i] = tr_join(ap[i]);
              }
              if constexpr (!BKM) {
#pragma unroll
                for (int j = 0; j < JN; ++j) bfr[j] = tr_join(bp[j]);
              }
            }
            mma_kk(af, bfr, sf, rf, sS, sR, kk);
          }
        };
        // strip rows past the used ones are never written: each only feeds
        // an MFMA result row of its own, which nothing reads
        if constexpr (NSTAGE == 1) {
          for (int kt = 0; kt < nk; ++kt) {
            if (PROT) issue_strip(kt);
            issue_dir(kt);
            if (PROT) issue_img(kt);
            wait_vmcnt<0>();
            if (PROT) commit_strip(kt);
            __syncthreads();
            compute_d(slot(kt));
            __syncthreads();
          }
        } else {
          static_assert(NSTAGE <= 2, "the strip image copy is waited for with vmcnt(0)");
          if (nk > 0 && PROT) issue_strip(0);
          for (int sl = 0; sl < NSTAGE - 1 && sl < nk; ++sl) {
            issue_dir(sl);
            if (PROT) issue_img(sl);
          }
          for (int kt = 0; kt < nk; ++kt) {
            // stage kt is complete once only the later stages' loads remain
            const int later = min(NSTAGE - 2, nk - 1 - kt);
            if (later >= 2) wait_vmcnt<(2 * NDIR < 63 ? 2 * NDIR : 63)>();
            else if (later == 1) wait_vmcnt<NDIR>();
            else wait_vmcnt<0>();
            if (PROT) commit_strip(kt);
            __syncthreads();  // stage kt visible; every wave is done with stage kt - 1
            if (PROT && kt + 1 < nk) issue_strip(kt + 1);
            if (kt + NSTAGE - 1 < nk) {
              issue_dir(kt + NSTAGE - 1);
              if (PROT) issue_img(kt + NSTAGE - 1);
            }
            compute_d(slot(kt));
          }
          __syncthreads();  // the epilogue reuses the stages
        }
      }
    } else {
    if (nk > 0) {
      la.load(A, g.lda, m0, g.M, k_lo, k_hi, tid);
      lb.load(B, g.ldb, n0, g.N, k_lo, k_hi, tid);
      if (cc) ls.load(Ac, g.ldac, rc0, nc_valid, k_lo, k_hi, tid);
      if (cr) lr.load(Br, g.ldbr, qc0, nq_valid, k_lo, k_hi, tid);
      la.store(lds, tid);
      lb.store(lds + A_ELEMS, tid);
      if (cc) ls.store(lds + A_ELEMS + B_ELEMS, nc, tid);
      if (cr) lr.store(lds + A_ELEMS + B_ELEMS + r_off, nq, tid);
      __syncthreads();
    }

    for (int kt = 0; kt < nk; ++kt) {
      const int cur = NSTAGE >= 2 ? (kt & 1) : 0;
      const bool more = kt + 1 < nk;
      if (more) {
        const int kn = k_lo + (kt + 1) * BK;
        la.load(A, g.lda, m0, g.M, kn, k_hi, tid);
        lb.load(B, g.ldb, n0, g.N, kn, k_hi, tid);
        if (cc) ls.load(Ac, g.ldac, rc0, nc_valid, kn, k_hi, tid);
        if (cr) lr.load(Br, g.ldbr, qc0, nq_valid, kn, k_hi, tid);
      }
      const T* sA = lds + (NSTAGE >= 2 ? cur : 0) * STAGE;
      const T* sB = sA + A_ELEMS;
      const T* sS = sB + B_ELEMS;
      const T* sR = sS + r_off;
#pragma unroll
      for (int kk = 0; kk < BK; kk += KI) {
        typename Mfma<T>::frag af[IM], bfr[JN];
#pragma unroll
        for (int i = 0; i < IM; ++i)
          af[i] = Mfma<T>::load(sA + (wm * WM + i * 16 + fr) * LDK + kk + fk);
#pragma unroll
        for (int j = 0; j < JN; ++j)
          bfr[j] = Mfma<T>::load(sB + (wn * WN + j * 16 + fr) * LDK + kk + fk);
        Frag sf, rf;
        strip_frags(sA, sS, sR, kk, sf, rf);
        mma_kk(af, bfr, sf, rf, sS, sR, kk);
      }
      if (more) {
        if (NSTAGE == 1) __syncthreads();  // every wave is done reading the one stage
        T* nA = lds + (NSTAGE >= 2 ? (cur ^ 1) : 0) * STAGE;
        la.store(nA, tid);
        lb.store(nA + A_ELEMS, tid);
        if (cc) ls.store(nA + A_ELEMS + B_ELEMS, nc, tid);
        if (cr) lr.store(nA + A_ELEMS + B_ELEMS + r_off, nq, tid);
      }
      __syncthreads();
    }
    }  // register path

    // ---- epilogue ----
    {
    const GemmDesc& g = desc_reload(slot);  // not held across the main loop
    if constexpr (sizeof(TC) == 4) if (split) {
      // fp32 partials go straight from the accumulators to this slice; the
      // column-checksum strip is combined (hi + lo) through a small LDS
      // image that fits inside the freed operand stages
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int j = 0; j < JN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = m0 + wm * WM + i * 16 + (lane >> 4) * 4 + r;
            const int n = n0 + wn * WN + j * 16 + fr;
            if (m < g.M && n < g.N) C[int64_t(m) * g.ldc + n] = TC(acc[i][j][r]);
          }
      if (PROT && cc && g.Cc != nullptr) {
        float* CsL = reinterpret_cast<float*>(smem);
#pragma unroll
        for (int j = 0; j < JS; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            CsL[((lane >> 4) * 4 + r) * BN + wn * WN + (wm * JS + j) * 16 + fr] = accs[j][r];
        __syncthreads();
        float* Cc = g.Cc + b0 * g.sCc0 + b1 * g.sCc1 + int64_t(kslice) * g.sCck;
        const int ncb = BM >> __builtin_ctz(g.Rm);
        for (int v = tid; v < ncb * BN; v += NT) {
          const int blk = v / BN, n = v % BN;
          float c1, c2;
          if constexpr (sizeof(T) == 2) {
            c1 = CsL[(4 * blk) * BN + n] + CsL[(4 * blk + 1) * BN + n];
            c2 = CsL[(4 * blk + 2) * BN + n] + CsL[(4 * blk + 3) * BN + n];
          } else {
            c1 = CsL[(2 * blk) * BN + n];
            c2 = CsL[(2 * blk + 1) * BN + n];
          }
          if (m0 + blk * g.Rm < g.M && n0 + n < g.N) {
            Cc[int64_t(rc0 + 2 * blk) * g.ldcc + n0 + n] = c1;
            Cc[int64_t(rc0 + 2 * blk + 1) * g.ldcc + n0 + n] = c2;
          }
        }
      }
      return;
    }
    // 1. round to storage and stage the tile (and the strip results) in LDS
    TC* tile = reinterpret_cast<TC*>(smem);
    float* CsL = reinterpret_cast<float*>(smem + TILE_BYTES);
    float* RsL = CsL + 16 * BN;
    float* ccv = CsL;         // after the strips are read
    float* rcv = ccv + CCV;
    float* colp = rcv + RCV;  // segment sums [BM / MINB][BN][2]
    float* rowp = colp + CCV; //              [BN / MINB][BM][2]
    // bf16 tiles take their segment sums on the matrix cores: the stored
    // values, packed two per register, are the MFMA operands
    uint32_t pk[MSUM ? IM : 1][MSUM ? JN : 1][2];
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int j = 0; j < JN; ++j) {
        const int row = wm * WM + i * 16 + (lane >> 4) * 4, col = wn * WN + j * 16 + fr;
        if constexpr (MSUM) {
          bf16_t h[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            h[r] = f2bf(acc[i][j][r]);
            tile[(row + r) * LDT + col] = h[r];
          }
          pk[i][j][0] = uint32_t(h[0]) | (uint32_t(h[1]) << 16);
          pk[i][j][1] = uint32_t(h[2]) | (uint32_t(h[3]) << 16);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)  // fp32 partials stay unrounded
            tile[(row + r) * LDT + col] = Storage<TC>::store(acc[i][j][r]);
        }
      }
    if (PROT && cc && !WLC) {
#pragma unroll
      for (int j = 0; j < JS; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          CsL[((lane >> 4) * 4 + r) * BN + wn * WN + (wm * JS + j) * 16 + fr] =
              accs[j][r];
    }
    if (PROT && cr && !WLC) {
#pragma unroll
      for (int i = 0; i < IS; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          RsL[(wm * WM + (wn * IS + i) * 16 + fr) * 16 + (lane >> 4) * 4 + r] =
              accr[i][r];
    }
    // injected faults (test-only): written into the rounded tile before any
    // verification
    if (wf) {
      __syncthreads();
      if (tid == 0) {
        for (int f = 0; f < g.n_faults; ++f) {
          const abft_fault ft = g.faults[f];
          int fz, fm, fn;
          if (fault_target(g.map, g.N, ft, &fz, &fm, &fn) && fz == z && fm >= m0 &&
              fm < m0 + BM && fn >= n0 && fn < n0 + BN)
            tile[(fm - m0) * LDT + fn - n0] =
                ft.mode == ABFT_FAULT_FLIP
                    ? flip_exponent_msb(tile[(fm - m0) * LDT + fn - n0])
                    : Storage<TC>::store(Storage<TC>::round(ft.value));
        }
      }
      __syncthreads();
      if constexpr (MSUM) {  // the packed values follow the tile
#pragma unroll
        for (int i = 0; i < IM; ++i)
#pragma unroll
          for (int j = 0; j < JN; ++j) {
            const TC* t = tile + (wm * WM + i * 16 + (lane >> 4) * 4) * LDT + wn * WN + j * 16 + fr;
            pk[i][j][0] = uint32_t(t[0]) | (uint32_t(t[LDT]) << 16);
            pk[i][j][1] = uint32_t(t[2 * LDT]) | (uint32_t(t[3 * LDT]) << 16);
          }
      }
    }
    if constexpr (WLC) {
      static_assert(MSUM, "the wave-local check is for protected bf16 tiles");
      epilogue_wlc(g, tile, A, B, C, z, b0, b1, m0, n0, k_lo, k_hi, cc, cr, rc0, qc0, pk, accs, accr,
                   reinterpret_cast<float*>(smem + TILE_BYTES), tid, slot);
      return;
    }
    __syncthreads();

    // 2. detection (Sec. 2.3 rule): recomputed against propagated checksums
    const int verify = (PROT && cc && !split) ? g.verify : 0;
    const int nrb = cr ? BN >> __builtin_ctz(g.Rn) : 0;   // row blocks per tile row
    const int ncb = cc ? BM >> __builtin_ctz(g.Rm) : 0;   // column blocks per tile column
    if (PROT && (cc || cr)) {
      // 2a. propagated checksums of every vector (strip hi + lo rows), held
      //     in registers until every thread has read the strips; row
      //     vectors are walked row-fastest, so only shifts divide
      constexpr int CI = int((CCV / 2 + NT - 1) / NT), RI = int((RCV / 2 + NT - 1) / NT);
      float2 cv[CI], rv[RI > 0 ? RI : 1];
#pragma unroll
      for (int i = 0; i < CI; ++i) {
        const int v = tid + i * NT, blk = v / BN, n = v % BN;
        if (v < ncb * BN) {
          if constexpr (sizeof(T) == 2) {
            cv[i].x = CsL[(4 * blk) * BN + n] + CsL[(4 * blk + 1) * BN + n];
            cv[i].y = CsL[(4 * blk + 2) * BN + n] + CsL[(4 * blk + 3) * BN + n];
          } else {
            cv[i].x = CsL[(2 * blk) * BN + n];
            cv[i].y = CsL[(2 * blk + 1) * BN + n];
          }
        }
      }
#pragma unroll
      for (int i = 0; i < RI; ++i) {
        const int w = tid + i * NT, row = w % BM, rb = w / BM;
        if (w < BM * nrb) {
          if constexpr (sizeof(T) == 2) {
            rv[i].x = RsL[row * 16 + 4 * rb] + RsL[row * 16 + 4 * rb + 1];
            rv[i].y = RsL[row * 16 + 4 * rb + 2] + RsL[row * 16 + 4 * rb + 3];
          } else {
            rv[i].x = RsL[row * 16 + 2 * rb];
            rv[i].y = RsL[row * 16 + 2 * rb + 1];
          }
        }
      }
      __syncthreads();  // the strip images are consumed; their space is reused
#pragma unroll
      for (int i = 0; i < CI; ++i)
        if (tid + i * NT < ncb * BN) reinterpret_cast<float2*>(ccv)[tid + i * NT] = cv[i];
#pragma unroll
      for (int i = 0; i < RI; ++i) {
        const int w = tid + i * NT;
        if (w < BM * nrb) reinterpret_cast<float2*>(rcv)[(w % BM) * nrb + w / BM] = rv[i];
      }
      // 2b. sums and magnitude sums of the stored tile over SEG-element
      //     segments
      constexpr int SEG = MINB;
      if constexpr (MSUM) {
        // A ones operand sums the k extent of the other operand, whatever
        // the order of k within it. Column segments: the 8 values of one
        // column a lane holds for blocks i = 2s, 2s + 1 (rows 4g..4g+3 of
        // each, g = lane / 16) are together the 32 rows of segment s.
        const bf16x8 ones = __builtin_bit_cast(
            bf16x8, uint4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});
        const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
        if (verify >= 1) {
#pragma unroll
          for (int sg = 0; sg < IM / 2; ++sg)
#pragma unroll
            for (int j = 0; j < JN; ++j) {
              const uint4 u = {pk[2 * sg][j][0], pk[2 * sg][j][1], pk[2 * sg + 1][j][0],
                               pk[2 * sg + 1][j][1]};
              const uint4 ua = {u.x & 0x7fff7fffu, u.y & 0x7fff7fffu, u.z & 0x7fff7fffu,
                                u.w & 0x7fff7fffu};
              const floatx4 sm = Mfma<T>::mma(ones, __builtin_bit_cast(bf16x8, u), zero);
              const floatx4 mg = Mfma<T>::mma(ones, __builtin_bit_cast(bf16x8, ua), zero);
              if (lane < 16)
                reinterpret_cast<float2*>(colp)[(wm * (WM / SEG) + sg) * BN + wn * WN + j * 16 +
                                                lane] = float2{sm[0], mg[0]};
            }
        }
        // row segments: 16 rows x 32 columns of the staged tile as the
        // A operand (row lane % 16, 8 consecutive columns per lane group);
        // lanes 0, 16, 32, 48 receive the sums of rows 4g..4g+3
        if (verify == 2) {
          constexpr int RG = BM / 16, UNITS = RG * (BN / SEG);
          static_assert(UNITS % (NT / 64) == 0, "row units per wave");
#pragma unroll
          for (int q = 0; q < UNITS / (NT / 64); ++q) {
            const int unit = wave * (UNITS / (NT / 64)) + q;
            const int r0 = (unit % RG) * 16, sg = unit / RG;
            const uint4 u = *reinterpret_cast<const uint4*>(
                tile + (r0 + (lane & 15)) * LDT + sg * SEG + 8 * (lane >> 4));
            const uint4 ua = {u.x & 0x7fff7fffu, u.y & 0x7fff7fffu, u.z & 0x7fff7fffu,
                              u.w & 0x7fff7fffu};
            const floatx4 sm = Mfma<T>::mma(__builtin_bit_cast(bf16x8, u), ones, zero);
            const floatx4 mg = Mfma<T>::mma(__builtin_bit_cast(bf16x8, ua), ones, zero);
            if ((lane & 15) == 0) {
              float4* o = reinterpret_cast<float4*>(rowp + (sg * BM + r0 + 4 * (lane >> 4)) * 2);
              o[0] = float4{sm[0], mg[0], sm[1], mg[1]};
              o[1] = float4{sm[2], mg[2], sm[3], mg[3]};
            }
          }
        }
      } else {
        // column pairs read 4 (or 8) bytes per row, row segments 16 bytes
        // at a time, so every thread has a share
        if (verify >= 1) {
          for (int w = tid; w < (BN / 2) * (BM / SEG); w += NT) {
            const int cp = w % (BN / 2), sg = w / (BN / 2);
            const TC* p = tile + sg * SEG * LDT + 2 * cp;
            float s0 = 0.f, s1 = 0.f, a0 = 0.f, a1 = 0.f;
#pragma unroll 8
            for (int r = 0; r < SEG; ++r) {
              float x0, x1;
              if constexpr (sizeof(TC) == 2) {
                const uint32_t wd = *reinterpret_cast<const uint32_t*>(p + r * LDT);
                x0 = __uint_as_float(wd << 16);
                x1 = __uint_as_float(wd & 0xffff0000u);
              } else {
                const float2 f = *reinterpret_cast<const float2*>(p + r * LDT);
                x0 = f.x;
                x1 = f.y;
              }
              s0 += x0; s1 += x1;
              a0 += fabsf(x0); a1 += fabsf(x1);
            }
            float* o = colp + (sg * BN + 2 * cp) * 2;
            o[0] = s0; o[1] = a0; o[2] = s1; o[3] = a1;
          }
        }
        if (verify == 2) {
          constexpr int PER16 = 16 / sizeof(TC);
          for (int w = tid; w < BM * (BN / SEG); w += NT) {
            const int row = w % BM, sg = w / BM;
            const TC* p = tile + row * LDT + sg * SEG;
            float s0 = 0.f, a0 = 0.f;
#pragma unroll
            for (int q = 0; q < SEG / PER16; ++q) {
              const uint4 raw = *reinterpret_cast<const uint4*>(p + q * PER16);
              const uint32_t wd[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
              for (int k = 0; k < 4; ++k) {
                if constexpr (sizeof(TC) == 2) {
                  const float x0 = __uint_as_float(wd[k] << 16);
                  const float x1 = __uint_as_float(wd[k] & 0xffff0000u);
                  s0 += x0 + x1;
                  a0 += fabsf(x0) + fabsf(x1);
                } else {
                  const float x0 = __uint_as_float(wd[k]);
                  s0 += x0;
                  a0 += fabsf(x0);
                }
              }
            }
            rowp[w * 2] = s0;
            rowp[w * 2 + 1] = a0;
          }
        }
      }
      __syncthreads();
      // 2c. decisions: one per checksum vector from its segments
      bool my_flag = false;
      if (verify >= 1) {
        const int spb = g.Rm / SEG;  // segments per column block
        for (int v = tid; v < ncb * BN; v += NT) {
          const int blk = v / BN, n = v % BN;
          if (!(m0 + blk * g.Rm < g.M && n0 + n < g.N && n0 + n >= g.verify_n_lo &&
                n0 + n < g.verify_n_hi))
            continue;
          float r1 = 0.f, sa = 0.f;
          for (int q = 0; q < spb; ++q) {
            r1 += colp[((blk * spb + q) * BN + n) * 2];
            sa += colp[((blk * spb + q) * BN + n) * 2 + 1];
          }
          my_flag |= flagged(ccv[v * 2] - r1, sa, g.e_rel);
        }
      }
      if (verify == 2) {
        const int spb = g.Rn / SEG;  // segments per row block
        for (int w = tid; w < BM * nrb; w += NT) {
          const int row = w % BM, rb = w / BM;
          if (!(m0 + row < g.M && n0 + rb * g.Rn < g.N)) continue;
          float r1 = 0.f, sa = 0.f;
          for (int q = 0; q < spb; ++q) {
            r1 += rowp[((rb * spb + q) * BM + row) * 2];
            sa += rowp[((rb * spb + q) * BM + row) * 2 + 1];
          }
          my_flag |= flagged(rcv[(row * nrb + rb) * 2] - r1, sa, g.e_rel);
        }
      }
      // 3. correction, only for a tile with a flagged vector
      if (__syncthreads_or(my_flag))
        passes(tile, A, B, z, m0, n0, k_lo, k_hi, ccv, rcv, reinterpret_cast<int*>(colp), nrb, ncb,
               verify, tid, slot);
    }

    // 4. store the tile with 16-byte coalesced chunks
    {
      constexpr int V = 16 / sizeof(TC);
      constexpr int CPR = BN / V;  // chunks per tile row
      for (int c = tid; c < BM * CPR; c += NT) {
        const int row = c / CPR, col = (c % CPR) * V;
        const int m = m0 + row, n = n0 + col;
        if (m >= g.M) continue;
        const TC* srcp = tile + row * LDT + col;
        TC* dstp = C + int64_t(m) * g.ldc + n;
        if (n + V <= g.N) {
          *reinterpret_cast<uint4*>(dstp) = *reinterpret_cast<const uint4*>(srcp);
        } else {
          for (int e = 0; e < V && n + e < g.N; ++e) dstp[e] = srcp[e];
        }
      }
    }

    // propagated checksums for the consumers downstream
    if (PROT && cc && g.Cc != nullptr) {
      float* Cc = g.Cc + b0 * g.sCc0 + b1 * g.sCc1 + int64_t(kslice) * g.sCck;
      for (int v = tid; v < ncb * BN; v += NT) {
        const int blk = v / BN, n = v % BN;
        if (m0 + blk * g.Rm < g.M && n0 + n < g.N) {
          Cc[int64_t(rc0 + 2 * blk) * g.ldcc + n0 + n] = ccv[v * 2];
          Cc[int64_t(rc0 + 2 * blk + 1) * g.ldcc + n0 + n] = ccv[v * 2 + 1];
        }
      }
    }
    if (PROT && cr && g.Cr != nullptr) {
      float* Cr = g.Cr + b0 * g.sCr0 + b1 * g.sCr1;
      for (int u = tid; u < BM * nrb; u += NT) {
        const int row = u / nrb, rb = u % nrb;
        if (m0 + row < g.M && n0 + rb * g.Rn < g.N) {
          Cr[int64_t(m0 + row) * g.ldcr + qc0 + 2 * rb] = rcv[u * 2];
          Cr[int64_t(m0 + row) * g.ldcr + qc0 + 2 * rb + 1] = rcv[u * 2 + 1];
        }
      }
    }
    }  // epilogue
  }

  // Wave-local column check (WLC): the wave holds every row of its WN
  // columns, so each column vector lies in the wave. Detection sums come
  // from ones-operand MFMAs on the packed stored values (the 8 values of
  // one column a lane holds for blocks i = 2s, 2s + 1 are the 32 rows of
  // segment s); the propagated checksums of column block b are the strip
  // rows 4b..4b+3, i.e. lane group b of the strip result (hi/lo c1, c2).
  // The wave stores its part of the tile at once. A two-sided output also
  // checks its rows: each wave sums its 32-column segments of every row
  // (ones-operand MFMAs on the staged tile), the partial sums meet in LDS
  // behind one barrier, and the lanes holding a row's propagated row
  // checksums (lane group b of the row strip: row block b) decide it. A
  // tile with a flagged vector then takes the workgroup through the
  // correction passes and is stored again.
  __device__ static __forceinline__ void epilogue_wlc(
      const GemmDesc& g, TC* tile, const T* A, const T* B, TC* C, int z, int b0, int b1, int m0,
      int n0, int k_lo, int k_hi, bool cc, bool cr, int rc0, int qc0,
      const uint32_t (&pk)[IM][JN][2],
      const floatx4 (&accs)[JS], const floatx4 (&accr)[IS], float* region, int tid, int slot) {
    const int lane = tid & 63, wn = tid >> 6;
    const int fr = lane & 15, g4 = lane >> 4;
    constexpr int SEG = MINB;
    const int verify = cc ? g.verify : 0;
    // the wave reads back only what it wrote itself
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    const int lg_rm = cc ? __builtin_ctz(g.Rm) : 0;
    const bool own_c = cc && g4 < (BM >> lg_rm) && m0 + (g4 << lg_rm) < g.M;
    bool flag = false;
    if (verify >= 1) {
      const bf16x8 ones = __builtin_bit_cast(
          bf16x8, uint4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});
      const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < JN; ++j) {
        float r1 = 0.f, sa = 0.f;
#pragma unroll
        for (int sg = 0; sg < IM / 2; ++sg) {
          const uint4 u = {pk[2 * sg][j][0], pk[2 * sg][j][1], pk[2 * sg + 1][j][0],
                           pk[2 * sg + 1][j][1]};
          const uint4 ua = {u.x & 0x7fff7fffu, u.y & 0x7fff7fffu, u.z & 0x7fff7fffu,
                            u.w & 0x7fff7fffu};
          const floatx4 sm = Mfma<T>::mma(ones, __builtin_bit_cast(bf16x8, u), zero);
          const floatx4 mg = Mfma<T>::mma(ones, __builtin_bit_cast(bf16x8, ua), zero);
          if (((sg * SEG) >> lg_rm) == g4) {
            r1 += sm[0];
            sa += mg[0];
          }
        }
        const int n = n0 + wn * WN + j * 16 + fr;
        if (own_c && n < g.N && n >= g.verify_n_lo && n < g.verify_n_hi)
          flag |= flagged(accs[j][0] + accs[j][1] - r1, sa, g.e_rel);
      }
    }

    // store this wave's part: 16-byte chunks, WN / 8 lanes per row piece
    constexpr int V = 16 / sizeof(TC), CPW = WN / V;
    static_assert((WM * CPW) % 64 == 0, "whole wave passes");
    const int nrb = (cr && verify == 2) ? BN >> __builtin_ctz(g.Rn) : 0;  // row blocks per tile row
    // with four chunks per row piece (WN = 4 V) and whole SEG-column
    // segments, pass i stores rows 16 i + lane % 16 (lane group g4: chunk
    // g4), and the same 16 bytes are the B operand of the row sums of a
    // two-sided output: one LDS read for both
    constexpr bool ROWS_IN_STORE = WN == 4 * V && WN == SEG;
    // a score-shaped output (causal 1) leaves the chunks wholly above the
    // diagonal unwritten: no consumer reads them (the softmax selects masked
    // keys to zero whatever is stored)
    const bool tri = g.causal == 1;
    if constexpr (ROWS_IN_STORE) {
      const bf16x8 ones = __builtin_bit_cast(
          bf16x8, uint4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});
      const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
      float2* part = reinterpret_cast<float2*>(region);  // [BN / SEG][BM]
#pragma unroll
      for (int i = 0; i < IM; ++i) {
        const int row = i * 16 + fr, col = wn * WN + g4 * V;
        const int m = m0 + row, n = n0 + col;
        const TC* srcp = tile + row * LDT + col;
        const uint4 u = *reinterpret_cast<const uint4*>(srcp);
        if (m < g.M && !(tri && n > m)) {
          TC* dstp = C + int64_t(m) * g.ldc + n;
          if (n + V <= g.N) {
            *reinterpret_cast<uint4*>(dstp) = u;
          } else {
            for (int e = 0; e < V && n + e < g.N; ++e) dstp[e] = srcp[e];
          }
        }
        if (nrb > 0) {
          const uint4 ua = {u.x & 0x7fff7fffu, u.y & 0x7fff7fffu, u.z & 0x7fff7fffu,
                            u.w & 0x7fff7fffu};
          const floatx4 sm = Mfma<T>::mma(ones, __builtin_bit_cast(bf16x8, u), zero);
          const floatx4 mg = Mfma<T>::mma(ones, __builtin_bit_cast(bf16x8, ua), zero);
          if (g4 == 0) part[wn * BM + i * 16 + fr] = float2{sm[0], mg[0]};
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < WM * CPW / 64; ++q) {
        const int c = lane + q * 64;
        const int row = c / CPW, col = wn * WN + (c % CPW) * V;
        const int m = m0 + row, n = n0 + col;
        if (m < g.M && !(tri && n > m)) {
          const TC* srcp = tile + row * LDT + col;
          TC* dstp = C + int64_t(m) * g.ldc + n;
          if (n + V <= g.N) {
            *reinterpret_cast<uint4*>(dstp) = *reinterpret_cast<const uint4*>(srcp);
          } else {
            for (int e = 0; e < V && n + e < g.N; ++e) dstp[e] = srcp[e];
          }
        }
      }
    }
    // propagated checksums for the consumers downstream (a correction
    // changes the output, not its propagated checksums)
    if (cc && g.Cc != nullptr && own_c) {
      float* Cc = g.Cc + b0 * g.sCc0 + b1 * g.sCc1;
#pragma unroll
      for (int j = 0; j < JN; ++j) {
        const int n = n0 + wn * WN + j * 16 + fr;
        if (n < g.N) {
          Cc[int64_t(rc0 + 2 * g4) * g.ldcc + n] = accs[j][0] + accs[j][1];
          Cc[int64_t(rc0 + 2 * g4 + 1) * g.ldcc + n] = accs[j][2] + accs[j][3];
        }
      }
    }
    if (cr && g.Cr != nullptr) {
      const int nrb = BN >> __builtin_ctz(g.Rn);
      if (g4 < nrb && n0 + g4 * g.Rn < g.N) {
        float* Cr = g.Cr + b0 * g.sCr0 + b1 * g.sCr1;
#pragma unroll
        for (int i = 0; i < IS; ++i) {
          const int m = m0 + (IS * wn + i) * 16 + fr;
          if (m < g.M) {
            Cr[int64_t(m) * g.ldcr + qc0 + 2 * g4] = accr[i][0] + accr[i][1];
            Cr[int64_t(m) * g.ldcr + qc0 + 2 * g4 + 1] = accr[i][2] + accr[i][3];
          }
        }
      }
    }
    if constexpr (WN % SEG == 0) {
      if (nrb > 0) {
        // partial sums of each row over this wave's SEG-column segments:
        // the staged rows as the B operand (column = row lane % 16, 8
        // consecutive columns per lane group), so every lane gets a row sum
        // (taken with the store above when the wave's columns are one
        // segment)
        constexpr int TS = WN / SEG;                 // segments per wave
        float2* part = reinterpret_cast<float2*>(region);  // [BN / SEG][BM]
        if constexpr (!ROWS_IN_STORE) {
          const bf16x8 ones = __builtin_bit_cast(
              bf16x8, uint4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});
          const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int i = 0; i < IM; ++i)
#pragma unroll
            for (int t = 0; t < TS; ++t) {
              const uint4 u = *reinterpret_cast<const uint4*>(
                  tile + (i * 16 + fr) * LDT + wn * WN + t * SEG + 8 * g4);
              const uint4 ua = {u.x & 0x7fff7fffu, u.y & 0x7fff7fffu, u.z & 0x7fff7fffu,
                                u.w & 0x7fff7fffu};
              const floatx4 sm = Mfma<T>::mma(ones, __builtin_bit_cast(bf16x8, u), zero);
              const floatx4 mg = Mfma<T>::mma(ones, __builtin_bit_cast(bf16x8, ua), zero);
              if (g4 == 0) part[(wn * TS + t) * BM + i * 16 + fr] = float2{sm[0], mg[0]};
            }
        }
        __syncthreads();
        // lane group g4 of the row strip holds row block g4 of rows
        // (IS wn + i) 16 + lane % 16
        const int spb = g.Rn / SEG;
        if (g4 < nrb && n0 + g4 * g.Rn < g.N) {
#pragma unroll
          for (int i = 0; i < IS; ++i) {
            const int row = (IS * wn + i) * 16 + fr;
            if (m0 + row < g.M) {
              float r1 = 0.f, sa = 0.f;
              for (int q = 0; q < spb; ++q) {
                const float2 pq = part[(g4 * spb + q) * BM + row];
                r1 += pq.x;
                sa += pq.y;
              }
              flag |= flagged(accr[i][0] + accr[i][1] - r1, sa, g.e_rel);
            }
          }
        }
      }
    }
    if (!__syncthreads_or(flag)) return;

    // a flagged vector: the checksums go to LDS in the layout of the
    // correction passes; the workgroup corrects and stores the tile again
    const int ncb = cc ? BM >> lg_rm : 0;
    float* ccv = region;
    float* rcv = ccv + CCV;
    int* work = reinterpret_cast<int*>(rcv + RCV);
    if (own_c) {
#pragma unroll
      for (int j = 0; j < JN; ++j) {
        const int v = g4 * BN + wn * WN + j * 16 + fr;
        ccv[v * 2] = accs[j][0] + accs[j][1];
        ccv[v * 2 + 1] = accs[j][2] + accs[j][3];
      }
    }
    if (g4 < nrb) {
#pragma unroll
      for (int i = 0; i < IS; ++i) {
        const int u = ((IS * wn + i) * 16 + fr) * nrb + g4;
        rcv[u * 2] = accr[i][0] + accr[i][1];
        rcv[u * 2 + 1] = accr[i][2] + accr[i][3];
      }
    }
    __syncthreads();
    passes(tile, A, B, z, m0, n0, k_lo, k_hi, ccv, rcv, work, nrb, ncb, verify, tid, slot);
    for (int c = tid; c < BM * (BN / V); c += NT) {
      const int row = c / (BN / V), col = (c % (BN / V)) * V;
      const int m = m0 + row, n = n0 + col;
      if (m >= g.M) continue;
      const TC* srcp = tile + row * LDT + col;
      TC* dstp = C + int64_t(m) * g.ldc + n;
      if (n + V <= g.N) {
        *reinterpret_cast<uint4*>(dstp) = *reinterpret_cast<const uint4*>(srcp);
      } else {
        for (int e = 0; e < V && n + e < g.N; ++e) dstp[e] = srcp[e];
      }
    }
    if (nrb > 0) {  // checksums the passes refreshed (1R / 1C) go downstream
      if (cc && g.Cc != nullptr) {
        float* Cc = g.Cc + b0 * g.sCc0 + b1 * g.sCc1;
        for (int v = tid; v < ncb * BN; v += NT) {
          const int blk = v / BN, n = v % BN;
          if (m0 + blk * g.Rm < g.M && n0 + n < g.N) {
            Cc[int64_t(rc0 + 2 * blk) * g.ldcc + n0 + n] = ccv[v * 2];
            Cc[int64_t(rc0 + 2 * blk + 1) * g.ldcc + n0 + n] = ccv[v * 2 + 1];
          }
        }
      }
      if (g.Cr != nullptr) {
        float* Cr = g.Cr + b0 * g.sCr0 + b1 * g.sCr1;
        for (int u = tid; u < BM * nrb; u += NT) {
          const int row = u / nrb, rb = u % nrb;
          if (m0 + row < g.M && n0 + rb * g.Rn < g.N) {
            Cr[int64_t(m0 + row) * g.ldcr + qc0 + 2 * rb] = rcv[u * 2];
            Cr[int64_t(m0 + row) * g.ldcr + qc0 + 2 * rb + 1] = rcv[u * 2 + 1];
          }
        }
      }
    }
  }

  // EEC-ABFT on the LDS tile, one thread per vector (as in the paper's
  // Fig. 4): column pass, refresh of 1R-corrupted row checksums, row pass,
  // refresh of 1C-corrupted column checksums, final check (Sec. 4.2, 4.3).
  __device__ static __forceinline__ void passes(
      TC* tile, const T* A, const T* B, int z, int m0, int n0, int k_lo, int k_hi, float* ccv,
      float* rcv, int* work, int nrb, int ncb, int verify, int tid, int slot) {
    const GemmDesc& g = desc_reload(slot);
    int* rowcnt = work;                        // [BM][BN / MINB]
    int* colcnt = work + BM * (BN / MINB);     // [BM / MINB][BN]
    for (int e = tid; e < int(CNT); e += NT) rowcnt[e] = 0;
    int* qn = work + CNT;                      // queue length
    int* qe = qn + 1;                                         // queue entries
    float* red = reinterpret_cast<float*>(qe + 3 * QMAX);     // per-wave partials
    if (tid == 0) *qn = 0;
    __syncthreads();
    const int Rm = g.Rm, Rn = g.Rn;
    const int lane = tid & 63, wave = tid >> 6;
    auto in_col = [&](int blk, int n) {
      return m0 + blk * Rm < g.M && n0 + n < g.N && n0 + n >= g.verify_n_lo &&
             n0 + n < g.verify_n_hi;
    };
    auto in_row = [&](int row, int rb) { return m0 + row < g.M && n0 + rb * Rn < g.N; };
    // A located element is recomputed from A and B by the whole workgroup
    // (its dot product split over the threads), so a correction costs a few
    // microseconds whatever K is: it is queued here and the queue is
    // drained after the pass. Corrections from the checksums alone are
    // applied at once.
    auto correct = [&](int lr, int lc, const TC* vec, int stride, int nvec, int idx, float c1,
                       float d1) {
      const float old = Storage<TC>::load(tile[lr * LDT + lc]);
      int action;
      float val;
      if (g.recompute) {
        const int slot = atomicAdd(qn, 1);
        if (slot < QMAX) {
          qe[3 * slot] = lr;
          qe[3 * slot + 1] = lc;
          qe[3 * slot + 2] = __float_as_int(old);
          return;
        }
        val = recompute_elem<T, TC, AK, BKM>(g, A, B, m0 + lr, n0 + lc, k_lo, k_hi);
        action = ABFT_ACT_RECOMPUTE;
      } else {
        val = fix_by_checksum<TC>(vec, stride, nvec, idx, c1, d1, g.tc, &action);
      }
      tile[lr * LDT + lc] = Storage<TC>::store(val);
      const EvCoord ec = map_coord(g.map, z, m0 + lr, n0 + lc);
      record_event(g.report, ec.op, ec.b, ec.h, ec.row, ec.col, classify(old, g.tn), action, old);
    };
    auto drain = [&]() {  // every thread of the workgroup
      __syncthreads();
      const int nq = min(*qn, QMAX);
      for (int q = 0; q < nq; ++q) {
        const int lr = qe[3 * q], lc = qe[3 * q + 1];
        const int m = m0 + lr, n = n0 + lc;
        float part = 0.f;
#pragma unroll 8
        for (int k = k_lo + tid; k < k_hi; k += NT)
          part = fmaf(Storage<T>::load(A[op_off<AK>(m, k, g.lda)]),
                      Storage<T>::load(B[op_off<BKM>(n, k, g.ldb)]), part);
        part = group_sum<64>(part);
        if (lane == 0) red[wave] = part;
        __syncthreads();
        if (tid == 0) {
          float val = 0.f;
          for (int w = 0; w < NT / 64; ++w) val += red[w];
          const float old = __int_as_float(qe[3 * q + 2]);
          tile[lr * LDT + lc] = Storage<TC>::store(val);
          const EvCoord ec = map_coord(g.map, z, m, n);
          record_event(g.report, ec.op, ec.b, ec.h, ec.row, ec.col, classify(old, g.tn),
                       ABFT_ACT_RECOMPUTE, old);
        }
        __syncthreads();
      }
      if (tid == 0) *qn = 0;
      __syncthreads();
    };

    // 1. column pass
    for (int v = tid; v < ncb * BN; v += NT) {
      const int blk = v / BN, n = v % BN;
      if (!in_col(blk, n)) continue;
      const TC* vec = tile + blk * Rm * LDT + n;
      const EecResult res = eec_locate<TC>(vec, LDT, Rm, ccv[v * 2], ccv[v * 2 + 1], g.e_rel, g.tn);
      if (res.status == EEC_LOCATED) {
        const int lr = blk * Rm + res.index;
        correct(lr, n, vec, LDT, Rm, res.index, ccv[v * 2], res.d1);
        if (verify == 2) atomicAdd(&rowcnt[lr * nrb + n / Rn], 1);
      }
    }
    drain();
    if (verify == 2) {
      // 2a. refresh row checksums of row vectors with >= 2 corrections (1R)
      for (int u = tid; u < BM * nrb; u += NT) {
        const int row = u / nrb, rb = u % nrb;
        if (in_row(row, rb) && rowcnt[u] >= 2)
          vec_checksums<TC>(tile + row * LDT + rb * Rn, 1, Rn, &rcv[u * 2], &rcv[u * 2 + 1]);
      }
      __syncthreads();
      // 2b. row pass
      for (int u = tid; u < BM * nrb; u += NT) {
        const int row = u / nrb, rb = u % nrb;
        if (!in_row(row, rb)) continue;
        const TC* vec = tile + row * LDT + rb * Rn;
        const EecResult res = eec_locate<TC>(vec, 1, Rn, rcv[u * 2], rcv[u * 2 + 1], g.e_rel, g.tn);
        if (res.status == EEC_LOCATED) {
          const int lc = rb * Rn + res.index;
          correct(row, lc, vec, 1, Rn, res.index, rcv[u * 2], res.d1);
          atomicAdd(&colcnt[(row / Rm) * BN + lc], 1);
        }
      }
      drain();
      // 2c. refresh column checksums of column vectors with >= 2 corrections (1C)
      for (int v = tid; v < ncb * BN; v += NT) {
        const int blk = v / BN, n = v % BN;
        if (in_col(blk, n) && colcnt[v] >= 2)
          vec_checksums<TC>(tile + blk * Rm * LDT + n, LDT, Rm, &ccv[v * 2], &ccv[v * 2 + 1]);
      }
      __syncthreads();
    }
    // 3. final check: anything still inconsistent is uncorrectable (2-D)
    for (int v = tid; v < ncb * BN; v += NT) {
      const int blk = v / BN, n = v % BN;
      if (!in_col(blk, n)) continue;
      if (vec_flagged<TC>(tile + blk * Rm * LDT + n, LDT, Rm, ccv[v * 2], g.e_rel)) {
        const EvCoord ec = map_coord(g.map, z, m0 + blk * Rm, n0 + n);
        record_event(g.report, ec.op, ec.b, ec.h, ec.row, ec.col, ABFT_KIND_NONE,
                     ABFT_ACT_UNCORRECTABLE, 0.f);
      }
    }
    if (verify == 2) {
      for (int u = tid; u < BM * nrb; u += NT) {
        const int row = u / nrb, rb = u % nrb;
        if (!in_row(row, rb)) continue;
        if (vec_flagged<TC>(tile + row * LDT + rb * Rn, 1, Rn, rcv[u * 2], g.e_rel)) {
          const EvCoord ec = map_coord(g.map, z, m0 + row, n0 + rb * Rn);
          record_event(g.report, ec.op, ec.b, ec.h, ec.row, ec.col, ABFT_KIND_NONE,
                       ABFT_ACT_UNCORRECTABLE, 0.f);
        }
      }
    }
    __syncthreads();
  }
};

// Tiles up to 128 x 128 keep two waves per SIMD (at most 256 registers,
// arch + accumulation, per lane), so two workgroups share a CU; the
// one-stage bf16 tile, which has no load in flight while it computes, keeps
// three (at most 168 registers) to hide its loads behind the other
// workgroups' work: unprotected, or protected with the wave-local check on
// the direct path (a few spills, far cheaper than the lost workgroup).
template <class T, int BM, int BN, bool PROT, int NSTAGE, bool WLC>
constexpr int gemm_waves_per_eu() {
  return BM * BN > 128 * 128 ? 1 : (sizeof(T) == 2 && NSTAGE == 1 && (!PROT || WLC) ? 3 : 2);
}

template <class T, class TC, bool AK, bool BKM, int BM, int BN, bool PROT, int NSTAGE, bool DIR,
          bool WLC>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(gemm_waves_per_eu<T, BM, BN, PROT, NSTAGE, WLC && DIR>())))
void gemm_kernel(GemmDesc g) {
  extern __shared__ __align__(16) char smem[];
  Gemm<T, TC, AK, BKM, BM, BN, PROT, NSTAGE, WLC>::template run<DIR>(g, smem, blockIdx.x,
                                                                      gridDim.x, 0);
}

// The direct-to-LDS path needs bf16 operands, K ranges of whole 64-wide
// stages (K a multiple of 64; causal K ranges and split-K slices then are
// too), 16-byte aligned operand rows, and whole 8-element chunks along the
// M or N extent of an MN-major operand.
template <class T>
bool direct_ok(const GemmDesc& g, bool ak, bool bk) {
  if (sizeof(T) != 2 || g.K % 64 != 0) return false;
  auto al = [](const void* p, int64_t ld, int64_t s0, int64_t s1) {
    return reinterpret_cast<uintptr_t>(p) % 16 == 0 && ld % 8 == 0 && s0 % 8 == 0 && s1 % 8 == 0;
  };
  if (!al(g.A, g.lda, g.sA0, g.sA1) || !al(g.B, g.ldb, g.sB0, g.sB1)) return false;
  if (!ak && (g.M % 8 != 0 || g.M < 8)) return false;
  if (!bk && (g.N % 8 != 0 || g.N < 8)) return false;
  return true;
}

// Sets the dynamic-LDS limit of one kernel once (per instantiation).
template <auto KERN>
hipError_t set_lds_limit(size_t bytes) {
  static bool done = false;  // harmless if repeated
  if (done) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(KERN),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, int(bytes));
  if (e == hipSuccess) done = true;
  return e;
}

template <class T, class TC, bool AK, bool BKM, int BM, int BN, bool PROT, int NSTAGE = 2>
hipError_t launch_t(const GemmDesc& g, hipStream_t s) {
  using G = Gemm<T, TC, AK, BKM, BM, BN, PROT, NSTAGE>;
  if (G::COLS_ONLY && (g.Br != nullptr || g.verify == 2)) return hipErrorInvalidValue;
  const bool gcc = PROT && g.Ac != nullptr, gcr = PROT && g.Br != nullptr;
  const bool direct = direct_ok<T>(g, AK, BKM);
  const size_t main = direct ? G::d_main_bytes(gcc, gcr) : G::main_bytes(gcc, gcr);
  // split-K slices skip the staged epilogue: only the operand stages (and
  // the 16 x BN checksum strip image inside them) are needed
  const size_t lds = g.splitk > 1 ? std::max(main, size_t(16 * BN * 4))
                                  : std::max(main, G::EPI_BYTES);
  const size_t lds_max = std::max(G::lds_bytes(PROT, PROT),
                                  sizeof(T) == 2 ? G::d_main_bytes(PROT, PROT) : size_t(0));
  if (lds_max > 160 * 1024) return hipErrorInvalidValue;  // this tile does not fit gfx950 LDS
  // wave-local column check for protected bf16 outputs verified on the
  // column side only (every checksum block of BM rows or less)
  bool wlc = false;
  // (two-sided outputs too when a wave's columns hold whole 32-column
  // segments)
  if constexpr (G::MSUM)
    wlc = g.splitk <= 1 && (g.verify <= 1 || BN / 4 >= 32) && (g.Ac == nullptr || g.Rm <= BM);
  auto kern = gemm_kernel<T, TC, AK, BKM, BM, BN, PROT, NSTAGE, false, false>;
  hipError_t e = hipSuccess;
  if constexpr (sizeof(T) == 2) {
    if (direct) {
      if constexpr (G::MSUM) {
        if (wlc) {
          constexpr auto k = gemm_kernel<T, TC, AK, BKM, BM, BN, PROT, NSTAGE, true, true>;
          kern = k;
          e = set_lds_limit<k>(lds_max);
        }
      }
      if (!wlc) {
        constexpr auto k = gemm_kernel<T, TC, AK, BKM, BM, BN, PROT, NSTAGE, true, false>;
        kern = k;
        e = set_lds_limit<k>(lds_max);
      }
    }
  }
  if (!direct) {
    if constexpr (G::MSUM) {
      if (wlc) {
        constexpr auto k = gemm_kernel<T, TC, AK, BKM, BM, BN, PROT, NSTAGE, false, true>;
        kern = k;
        e = set_lds_limit<k>(lds_max);
      }
    }
    if (!wlc) {
      constexpr auto k = gemm_kernel<T, TC, AK, BKM, BM, BN, PROT, NSTAGE, false, false>;
      e = set_lds_limit<k>(lds_max);
    }
  }
  if (e != hipSuccess) return e;
  const int64_t ntm = (g.M + BM - 1) / BM, ntn = (g.N + BN - 1) / BN;
  const int64_t tiles = tri_tiles(g, BM, BN) ? ntm * (ntm + 1) / 2 : ntm * ntn;
  const int64_t nb = int64_t(g.nb0) * g.nb1, ks = g.splitk > 1 ? g.splitk : 1;
  if (tiles == 0 || nb == 0) return hipSuccess;
  if (nb > 1 && ks > 1) return hipErrorInvalidValue;  // split-K is for unbatched GEMMs
  if (ks > 1 && sizeof(TC) != 4) return hipErrorInvalidValue;  // fp32 partial slices
  const int64_t total = tiles * nb * ks;
  if (total > 0x7fffffff / NT) return hipErrorInvalidValue;
  hipLaunchKernelGGL(kern, dim3(unsigned(total)), dim3(NT), lds, s, g);
  return hipGetLastError();
}

// Two independent GEMMs of the layer's backward in one launch: workgroups
// [0, n1) run a weight gradient (MN-major operands, fp32 output, whole or
// in K slices: the longer work items first), the rest a projection with
// K-major operands and bf16 output; both 128 x 128 tiles on the direct
// path. Alone, each leaves CUs idle in its last round of workgroups.
template <bool PROT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2)))
void gemm_pair_kernel(GemmDesc gw, GemmDesc gp, int n1) {
  extern __shared__ __align__(16) char smem[];
  if (int(blockIdx.x) < n1)
    Gemm<bf16_t, float, false, false, 128, 128, PROT, 2, false>::template run<true>(
        gw, smem, blockIdx.x, n1, 0);
  else
    Gemm<bf16_t, bf16_t, true, true, 128, 128, PROT, 2, PROT>::template run<true>(
        gp, smem, int(blockIdx.x) - n1, int(gridDim.x) - n1, 1);
}

template <bool PROT>
hipError_t pair_t(const GemmDesc& w, const GemmDesc& p, hipStream_t s) {
  using GW = Gemm<bf16_t, float, false, false, 128, 128, PROT, 2, false>;
  using GP = Gemm<bf16_t, bf16_t, true, true, 128, 128, PROT, 2, PROT>;
  if (!direct_ok<bf16_t>(w, false, false) || !direct_ok<bf16_t>(p, true, true))
    return hipErrorNotSupported;
  if (w.nb0 * w.nb1 != 1 || p.nb0 * p.nb1 != 1 || p.splitk > 1 || w.causal != 0 ||
      p.causal != 0)
    return hipErrorNotSupported;
  if (w.Br != nullptr || w.verify == 2) return hipErrorInvalidValue;  // columns only
  // the projection's epilogue as a launch of its own would take it: the
  // wave-local check when protected
  if (PROT && !((p.verify <= 1 || 128 / 4 >= 32) && (p.Ac == nullptr || p.Rm <= 128)))
    return hipErrorNotSupported;
  const bool wcc = PROT && w.Ac != nullptr, pcc = PROT && p.Ac != nullptr;
  const bool pcr = PROT && p.Br != nullptr;
  const size_t lw = w.splitk > 1 ? std::max(GW::d_main_bytes(wcc, false), size_t(16 * 128 * 4))
                                 : std::max(GW::d_main_bytes(wcc, false), GW::EPI_BYTES);
  const size_t lp = std::max(GP::d_main_bytes(pcc, pcr), GP::EPI_BYTES);
  const size_t lds = std::max(lw, lp);
  const size_t lds_max =
      std::max(std::max(GW::lds_bytes(PROT, PROT), GW::d_main_bytes(PROT, PROT)),
               std::max(GP::lds_bytes(PROT, PROT), GP::d_main_bytes(PROT, PROT)));
  if (lds_max > 160 * 1024) return hipErrorNotSupported;
  const int64_t ksw = w.splitk > 1 ? w.splitk : 1;
  const int64_t n1 = ((w.M + 127) / 128) * ((w.N + 127) / 128) * ksw;
  const int64_t n2 = ((p.M + 127) / 128) * ((p.N + 127) / 128);
  if (n1 == 0 || n2 == 0 || n1 % 8 != 0) return hipErrorNotSupported;  // keeps the XCD dealing
  if (n1 + n2 > 0x7fffffff / NT) return hipErrorInvalidValue;
  constexpr auto k = gemm_pair_kernel<PROT>;
  hipError_t e = set_lds_limit<k>(lds_max);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k, dim3(unsigned(n1 + n2)), dim3(NT), lds, s, w, p, int(n1));
  return hipGetLastError();
}

// The (layout, tile) pairs the attention layer launches; bf16 GEMMs with
// fp32 output are the split-K weight gradients only.
template <class T, class TC, bool AK, bool BKM, bool PROT>
hipError_t launch_tile(const GemmDesc& g, Tile tile, hipStream_t s) {
  constexpr bool wgrad = sizeof(T) == 2 && sizeof(TC) == 4;
  if constexpr (wgrad) {
    if constexpr (!AK && !BKM)
      if (tile == Tile::T128x128) return launch_t<T, TC, AK, BKM, 128, 128, PROT>(g, s);
    return hipErrorInvalidValue;
  } else {
    if (tile == Tile::T128x128) return launch_t<T, TC, AK, BKM, 128, 128, PROT>(g, s);
    if constexpr (AK && BKM) {
      if (tile == Tile::T128x128S1) return launch_t<T, TC, AK, BKM, 128, 128, PROT, 1>(g, s);
    } else {
      if (tile == Tile::T128x64) return launch_t<T, TC, AK, BKM, 128, 64, PROT>(g, s);
    }
    return hipErrorInvalidValue;
  }
}

template <class T, class TC, bool PROT>
hipError_t launch_layout(const GemmDesc& g, Layout la, Layout lb, Tile tile, hipStream_t s) {
  const bool ak = la == Layout::KMajor, bk = lb == Layout::KMajor;
  if (ak && !bk) return launch_tile<T, TC, true, false, PROT>(g, tile, s);
  if (ak && bk) return launch_tile<T, TC, true, true, PROT>(g, tile, s);
  if (!ak && !bk) return launch_tile<T, TC, false, false, PROT>(g, tile, s);
  return hipErrorInvalidValue;  // (MN-major A, K-major B) is not used by the layer
}

// Split-K reduction fused with the column check. One workgroup owns a
// block of RB rows (the checksum block, Rm rows, when verifying) and 32
// columns; each thread sums the K slices of one float4 column quad for
// every 32nd row of the block in a fixed order (deterministic), keeps the
// block in LDS and accumulates the columns' sums and magnitude sums. The
// row groups' partials of a column are combined in LDS; its checksums are
// the fixed-order sums of the slices' checksum rows. A flagged column runs EEC-ABFT (Sec. 4.2) on the LDS block
// with recompute correction and the final check; then the block is stored.
constexpr int RED_CQ = 8;  // float4 quads per workgroup row piece (more workgroups than 16)

// CQ quads (RED_COLS = 4 CQ columns) per workgroup, 256 / CQ row groups,
// RPT rows per thread (block of RB rows), KS slices; all fixed at compile
// time so that every load of a thread is in flight at once.
template <class T, bool AK, bool BKM, int RPT, int KS, int CQ>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmDesc g, const float* P,
                                                            const float* Pc, int verify) {
  constexpr int RED_COLS = 4 * CQ, RED_GROUPS = 256 / CQ;
  constexpr int SG = 256 / RED_COLS;                // slice groups of the checksum rows
  constexpr int RB = RPT * RED_GROUPS;
  __shared__ float blk[RB * RED_COLS];              // the reduced block
  __shared__ float p1[RED_GROUPS * RED_COLS], p2[RED_GROUPS * RED_COLS];
  __shared__ float pc[2][SG][RED_COLS];             // checksum partials per slice group
  const int cq = threadIdx.x % CQ, rg = threadIdx.x / CQ;
  const int c0 = cq * 4, n = blockIdx.x * RED_COLS + c0;
  const int rb = blockIdx.y, m_base = rb * RB;
  const int64_t MN = int64_t(g.M) * g.N;
  const bool col_ok = n < g.N;  // N % 4 == 0: a quad is all in or all out
  // whether an injected fault (test-only) lands in this workgroup's block
  bool wf = false;
  for (int f = 0; f < g.n_faults; ++f) {
    int fz, fm, fn;
    wf |= fault_target(g.map, g.N, g.faults[f], &fz, &fm, &fn) && fm >= m_base &&
          fm < m_base + RB && fn >= int(blockIdx.x) * RED_COLS && fn < int(blockIdx.x + 1) * RED_COLS;
  }

  // checksum rows of the slices: thread (c, sg) sums slices sg, sg+SG, ...
  const bool chk = verify && m_base + RB <= g.M;
  if (chk) {
    const int c = threadIdx.x % RED_COLS, sg = threadIdx.x / RED_COLS;
    const int nc = blockIdx.x * RED_COLS + c;
    const int64_t slc = int64_t(2 * (g.M / g.Rm)) * g.N;
    const int ncc = min(nc, g.N - 1);  // loads stay unconditional (see below)
    float a1 = 0.f, a2 = 0.f;
#pragma unroll
    for (int sl = sg; sl < KS; sl += SG) {
      a1 += Pc[sl * slc + int64_t(2 * rb) * g.N + ncc];
      a2 += Pc[sl * slc + int64_t(2 * rb + 1) * g.N + ncc];
    }
    pc[0][sg][c] = a1;
    pc[1][sg][c] = a2;
  }

  // Every load is unconditional, from a clamped (valid) address, and out
  // of range values are dropped afterwards: a load under a divergent branch
  // makes the compiler wait for it at the join, one load at a time.
  float4 v[RPT];
#pragma unroll
  for (int u = 0; u < RPT; ++u) v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
  const int nclamp = min(n, g.N - 4);
#pragma unroll
  for (int sl = 0; sl < KS; ++sl)
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      const int m = min(m_base + rg + RED_GROUPS * u, g.M - 1);
      const float4 t = *reinterpret_cast<const float4*>(P + sl * MN + int64_t(m) * g.N + nclamp);
      v[u].x += t.x; v[u].y += t.y; v[u].z += t.z; v[u].w += t.w;
    }
#pragma unroll
  for (int u = 0; u < RPT; ++u)
    if (!col_ok || m_base + rg + RED_GROUPS * u >= g.M) v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
  float r1[4] = {0.f, 0.f, 0.f, 0.f}, sa[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < RPT; ++u) {
    const int rr = rg + RED_GROUPS * u, m = m_base + rr;
    float e[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
    for (int f = 0; wf && f < g.n_faults; ++f) {  // injected faults (tests only)
      int fz, fm, fn;
      if (col_ok && fault_target(g.map, g.N, g.faults[f], &fz, &fm, &fn) && fm == m &&
          fn >= n && fn < n + 4) {
#pragma unroll
        for (int w = 0; w < 4; ++w)
          if (fn == n + w)
            e[w] = g.faults[f].mode == ABFT_FAULT_FLIP ? flip_exponent_msb(e[w])
                                                       : g.faults[f].value;
      }
    }
    *reinterpret_cast<float4*>(blk + rr * RED_COLS + c0) = make_float4(e[0], e[1], e[2], e[3]);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      r1[w] += e[w];
      sa[w] += fabsf(e[w]);
    }
  }
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    p1[rg * RED_COLS + c0 + w] = r1[w];
    p2[rg * RED_COLS + c0 + w] = sa[w];
  }
  __syncthreads();
  // decisions (one thread per column); a located element is recomputed
  // over K by the whole workgroup afterwards, then its column is checked
  // again
  __shared__ int flag[RED_COLS], qrow[RED_COLS];
  __shared__ float qold[RED_COLS], wsum[4];
  const int c = threadIdx.x, nc = blockIdx.x * RED_COLS + c;
  float c1 = 0.f;
  if (c < RED_COLS) {
    flag[c] = 0;
    qrow[c] = -1;
  }
  if (chk && c < RED_COLS && nc < g.N) {
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int q = 0; q < RED_GROUPS; ++q) {
      s1 += p1[q * RED_COLS + c];
      s2 += p2[q * RED_COLS + c];
    }
    float c2 = 0.f;
#pragma unroll
    for (int q = 0; q < SG && q < KS; ++q) {
      c1 += pc[0][q][c];
      c2 += pc[1][q][c];
    }
    if (flagged(c1 - s1, s2, g.e_rel)) {
      flag[c] = 1;
      float* col = blk + c;
      const EecResult res = eec_locate<float>(col, RED_COLS, RB, c1, c2, g.e_rel, g.tn);
      if (res.status == EEC_LOCATED) {
        const int lr = res.index;
        const float old = col[lr * RED_COLS];
        if (g.recompute) {
          qrow[c] = lr;
          qold[c] = old;
        } else {
          int action;
          col[lr * RED_COLS] = fix_by_checksum<float>(col, RED_COLS, RB, lr, c1, res.d1, g.tc,
                                                      &action);
          const EvCoord ec = map_coord(g.map, 0, m_base + lr, nc);
          record_event(g.report, ec.op, ec.b, ec.h, ec.row, ec.col, classify(old, g.tn), action,
                       old);
        }
      }
    }
  }
  __syncthreads();
  for (int q = 0; q < RED_COLS; ++q) {  // uniform: every thread reads the same queue
    const int lr = qrow[q];
    if (lr < 0) continue;
    const int m = m_base + lr, n = blockIdx.x * RED_COLS + q;
    const T* A = static_cast<const T*>(g.A);
    const T* B = static_cast<const T*>(g.B);
    float part = 0.f;
#pragma unroll 8
    for (int k = threadIdx.x; k < g.K; k += 256)
      part = fmaf(Storage<T>::load(A[op_off<AK>(m, k, g.lda)]),
                  Storage<T>::load(B[op_off<BKM>(n, k, g.ldb)]), part);
    part = group_sum<64>(part);
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = part;
    __syncthreads();
    if (threadIdx.x == 0) {
      blk[lr * RED_COLS + q] = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
      const EvCoord ec = map_coord(g.map, 0, m, n);
      record_event(g.report, ec.op, ec.b, ec.h, ec.row, ec.col, classify(qold[q], g.tn),
                   ABFT_ACT_RECOMPUTE, qold[q]);
    }
    __syncthreads();
  }
  if (c < RED_COLS && flag[c] && vec_flagged<float>(blk + c, RED_COLS, RB, c1, g.e_rel)) {
    const EvCoord ec = map_coord(g.map, 0, m_base, nc);
    record_event(g.report, ec.op, ec.b, ec.h, ec.row, ec.col, ABFT_KIND_NONE,
                 ABFT_ACT_UNCORRECTABLE, 0.f);
  }
  __syncthreads();
  if (!col_ok) return;
  float* C = static_cast<float*>(g.C);
#pragma unroll
  for (int u = 0; u < RPT; ++u) {
    const int rr = rg + RED_GROUPS * u, m = m_base + rr;
    if (m < g.M)
      *reinterpret_cast<float4*>(C + int64_t(m) * g.ldc + n) =
          *reinterpret_cast<const float4*>(blk + rr * RED_COLS + c0);
  }
}

template <class T, int RPT, int KS>
hipError_t reduce_launch(const GemmDesc& g, const float* P, const float* Pc, int verify,
                         hipStream_t s) {
  constexpr int RED_COLS = 4 * RED_CQ, RB = RPT * (256 / RED_CQ);
  dim3 grid((g.N + RED_COLS - 1) / RED_COLS, (g.M + RB - 1) / RB);
  hipLaunchKernelGGL((splitk_reduce_kernel<T, false, false, RPT, KS, RED_CQ>), grid, dim3(256), 0,
                     s, g, P, Pc, verify);
  return hipGetLastError();
}

template <class T, int RPT>
hipError_t reduce_ks(const GemmDesc& g, const float* P, const float* Pc, int verify,
                     hipStream_t s) {
  switch (g.splitk) {
    case 2: return reduce_launch<T, RPT, 2>(g, P, Pc, verify, s);
    case 4: return reduce_launch<T, RPT, 4>(g, P, Pc, verify, s);
    case 8: return reduce_launch<T, RPT, 8>(g, P, Pc, verify, s);
    case 16: return reduce_launch<T, RPT, 16>(g, P, Pc, verify, s);
  }
  return hipErrorInvalidValue;
}

template <class T>
hipError_t reduce_t(const GemmDesc& g, const float* P, const float* Pc, Layout la, Layout lb,
                    hipStream_t s) {
  if (la != Layout::MNMajor || lb != Layout::MNMajor) return hipErrorInvalidValue;
  if (g.ldc < g.N || g.N % 4 != 0 || g.ldc % 4 != 0) return hipErrorInvalidValue;
  const int verify = (g.verify >= 1 && g.Ac != nullptr && Pc != nullptr) ? 1 : 0;
  // the checksum block is the row block
  const int RB = verify ? g.Rm : 64;
  if (verify && g.M % RB != 0) return hipErrorInvalidValue;
  constexpr int RG = 256 / RED_CQ;  // row groups
  static_assert(64 % RG == 0, "a 64-row block covers the row groups");
  if (RB == 64) return reduce_ks<T, 64 / RG>(g, P, Pc, verify, s);
  if (RB == 128) return reduce_ks<T, 128 / RG>(g, P, Pc, verify, s);
  return hipErrorInvalidValue;  // head dimensions 64 and 128 only
}

}  // namespace

hipError_t launch_splitk_reduce(const GemmDesc& g, const float* P, const float* Pc, int dtype,
                                Layout la, Layout lb, hipStream_t stream) {
  if (dtype == ABFT_FP32) return reduce_t<float>(g, P, Pc, la, lb, stream);
  return reduce_t<bf16_t>(g, P, Pc, la, lb, stream);
}

hipError_t launch_gemm_pair(const GemmDesc& w, const GemmDesc& p, int dtype,
                            hipStream_t stream) {
  auto pow2 = [](int x) { return x > 0 && (x & (x - 1)) == 0; };
  if (dtype != ABFT_BF16) return hipErrorNotSupported;
  if (!pow2(w.Rm) || !pow2(w.Rn) || !pow2(p.Rm) || !pow2(p.Rn)) return hipErrorInvalidValue;
  const bool pw = w.Ac != nullptr || w.Br != nullptr || w.verify != 0;
  const bool pp = p.Ac != nullptr || p.Br != nullptr || p.verify != 0;
  if (pw != pp) return hipErrorNotSupported;
  return pp ? pair_t<true>(w, p, stream) : pair_t<false>(w, p, stream);
}

hipError_t launch_gemm(const GemmDesc& g, int dtype, bool c_fp32, Layout la, Layout lb,
                       Tile tile, hipStream_t stream) {
  auto pow2 = [](int x) { return x > 0 && (x & (x - 1)) == 0; };
  if (!pow2(g.Rm) || !pow2(g.Rn)) return hipErrorInvalidValue;  // the kernels shift by them
  const bool prot = g.Ac != nullptr || g.Br != nullptr || g.verify != 0;
  if (dtype == ABFT_FP32) {
    return prot ? launch_layout<float, float, true>(g, la, lb, tile, stream)
                : launch_layout<float, float, false>(g, la, lb, tile, stream);
  }
  if (c_fp32)
    return prot ? launch_layout<bf16_t, float, true>(g, la, lb, tile, stream)
                : launch_layout<bf16_t, float, false>(g, la, lb, tile, stream);
  return prot ? launch_layout<bf16_t, bf16_t, true>(g, la, lb, tile, stream)
              : launch_layout<bf16_t, bf16_t, false>(g, la, lb, tile, stream);
}

}  // namespace abft
