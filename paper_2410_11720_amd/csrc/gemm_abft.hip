// Protected GEMM for gfx950: C = A B on MFMA 16x16x32 bf16 (or 16x16x4
// f32), with the ABFT checksums of paper Sec. 2.3 carried as extra MFMA
// tiles (the "packed operand" update of Sec. 4.6): the column checksums
// A^c of the tile's row blocks form a 16-row strip that is multiplied by
// the same B fragments (C^c = A^c B), and, for two-sided outputs, the row
// checksums B^r form a 16-column strip multiplied by the same A fragments
// (C^r = A B^r). fp32 checksums enter a bf16 MFMA as a hi + lo bf16 pair,
// so the propagated checksum keeps ~16 significant bits.
//
// The epilogue rounds the tile to storage, applies injected faults, and
// compares recomputed against propagated checksums with wavefront
// reductions (detection, Sec. 2.3). A clean tile is stored directly. A
// flagged tile takes the slow path in LDS: EEC-ABFT on every column vector
// (Sec. 4.2), and for two-sided outputs the row pass with the checksum
// refresh of Sec. 4.3, then a final check; located elements are recomputed
// from A and B (or corrected from the checksums when the operands are not
// trusted) and every action is appended to the device report.
#include "abft_internal.hpp"
#include "abft_device.hpp"

namespace abft {

namespace {

constexpr int NT = 256;  // threads per workgroup: 4 waves as 2 (M) x 2 (N)

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
    if constexpr (KMAJ) {
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
// for the tile, stored as NC hi rows and NC lo rows (bf16) or NC fp32 rows.
template <class T, bool KMAJ>
struct StripLoader {
  static constexpr int BK = Mfma<T>::BK;
  static constexpr int LDK = BK + Mfma<T>::PAD;
  static constexpr int PER = (16 * BK + NT - 1) / NT;
  float reg[PER];

  // rows r0 + r exist only for r < nvalid (the last tile may be ragged)
  __device__ void load(const float* base, int64_t ld, int r0, int nvalid, int k0, int kend,
                       int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int e = tid + p * NT;
      const int r = e / BK, k = e % BK;
      float v = 0.f;
      if (r < nvalid && k0 + k < kend) v = base[op_off<KMAJ>(r0 + r, k0 + k, ld)];
      reg[p] = v;
    }
  }
  __device__ void store(T* lds, int nc, int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int e = tid + p * NT;
      const int r = e / BK, k = e % BK;
      if (r < nc) {
        if constexpr (sizeof(T) == 2) {
          const bf16_t hi = f2bf(reg[p]);
          const bf16_t lo = f2bf(reg[p] - bf2f(hi));
          lds[r * LDK + k] = hi;
          lds[(nc + r) * LDK + k] = lo;
        } else {
          lds[r * LDK + k] = reg[p];
        }
      }
    }
  }
};

__device__ __forceinline__ float wsum16(float x) {  // sum over lanes with equal lane%16
  x += __shfl_xor(x, 16, 64);
  x += __shfl_xor(x, 32, 64);
  return x;
}
__device__ __forceinline__ float wsum_row(float x) {  // sum over the 16 lanes of a row
  x += __shfl_xor(x, 1, 64);
  x += __shfl_xor(x, 2, 64);
  x += __shfl_xor(x, 4, 64);
  x += __shfl_xor(x, 8, 64);
  return x;
}

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
  for (int k = k_lo; k < k_hi; ++k)
    s = fmaf(Storage<T>::load(A[op_off<AK>(m, k, g.lda)]),
             Storage<T>::load(B[op_off<BKM>(n, k, g.ldb)]), s);
  return s;
}

template <class T, class TC, bool AK, bool BKM, int BM, int BN, bool PROT>
struct Gemm {
  static constexpr int BK = Mfma<T>::BK;
  static constexpr int KI = Mfma<T>::KI;
  static constexpr int LDK = BK + Mfma<T>::PAD;
  static constexpr int WM = BM / 2, WN = BN / 2;
  static constexpr int IM = WM / 16, JN = WN / 16;
  static constexpr int JS = JN / 2, IS = IM / 2;  // strip blocks per wave
  static_assert(IM >= 2 && JN >= 2, "tile too small");
  static constexpr int FRAG = KI / 4;  // operand elements per lane

  // LDS map of the main loop (two stages)
  static constexpr int A_ELEMS = BM * LDK, B_ELEMS = BN * LDK, S_ELEMS = 16 * LDK;
  static constexpr int STAGE = A_ELEMS + B_ELEMS + (PROT ? 2 * S_ELEMS : 0);
  static constexpr size_t MAIN_BYTES = size_t(2) * STAGE * sizeof(T);
  // LDS map of the epilogue: region 0 (strip results and partial sums, later
  // the slow-path tile) then region 1 (combined checksums and counters).
  static constexpr size_t CSL = 16 * BN, RSL = BM * 16;
  static constexpr size_t COLP = (BM / 16) * BN * 3, ROWP = (BN / 16) * BM * 3;
  static constexpr size_t R0_PART = (CSL + RSL + COLP + ROWP) * 4;
  static constexpr size_t R0_TILE = size_t(BM) * BN * sizeof(TC);
  static constexpr size_t R0 = R0_PART > R0_TILE ? R0_PART : R0_TILE;
  static constexpr size_t CCV = (BM / 16) * BN * 2, RCV = BM * (BN / 16) * 2;
  static constexpr size_t CNT = BM * (BN / 16) + (BM / 16) * BN;
  static constexpr size_t EPI_BYTES = R0 + (CCV + RCV) * 4 + CNT * 4;
  static constexpr size_t LDS_BYTES =
      PROT ? (MAIN_BYTES > EPI_BYTES ? MAIN_BYTES : EPI_BYTES)
           : (MAIN_BYTES > R0_TILE ? MAIN_BYTES : R0_TILE);

  __device__ static __forceinline__ void run(const GemmDesc& g, char* smem) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int ntn = (g.N + BN - 1) / BN;
    const int mt = blockIdx.x / ntn, nt = blockIdx.x % ntn;
    const int m0 = mt * BM, n0 = nt * BN;
    const int z = blockIdx.y;
    const int b0 = z / g.nb1, b1 = z % g.nb1;
    if (g.causal == 1 && n0 > m0 + BM - 1) return;  // whole tile above the diagonal

    int k_lo = 0, k_hi = g.K;
    if (g.causal == 2) k_hi = min(g.K, m0 + BM);
    if (g.causal == 3) k_lo = min(g.K, m0);

    const T* A = static_cast<const T*>(g.A) + b0 * g.sA0 + b1 * g.sA1;
    const T* B = static_cast<const T*>(g.B) + b0 * g.sB0 + b1 * g.sB1;
    TC* C = static_cast<TC*>(g.C) + b0 * g.sC0 + b1 * g.sC1;

    const bool cc = PROT && g.Ac != nullptr;
    const bool cr = PROT && g.Br != nullptr && n0 >= g.cr_n_begin;
    const int nc = cc ? 2 * BM / g.Rm : 0;           // checksum rows of this tile
    const int nq = cr ? 2 * BN / g.Rn : 0;           // checksum cols of this tile
    const int rc0 = 2 * (m0 / g.Rm);
    const int qc0 = cr ? 2 * ((n0 - g.cr_n_begin) / g.Rn) : 0;
    const int nc_valid = cc ? min(nc, 2 * (g.M / g.Rm) - rc0) : 0;
    const int nq_valid = cr ? min(nq, 2 * ((g.N - g.cr_n_begin) / g.Rn) - qc0) : 0;
    const float* Ac = cc ? g.Ac + b0 * g.sAc0 + b1 * g.sAc1 : nullptr;
    const float* Br = cr ? g.Br + b0 * g.sBr0 + b1 * g.sBr1 : nullptr;

    T* lds = reinterpret_cast<T*>(smem);
    TileLoader<T, AK, BM> la;
    TileLoader<T, BKM, BN> lb;
    StripLoader<T, AK> ls;
    StripLoader<T, BKM> lr;

    floatx4 acc[IM][JN];
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int j = 0; j < JN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    floatx4 accs[JS], accr[IS];
#pragma unroll
    for (int j = 0; j < JS; ++j) accs[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < IS; ++i) accr[i] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int nk = k_hi > k_lo ? (k_hi - k_lo + BK - 1) / BK : 0;
    if (nk > 0) {
      if (PROT) {  // zero both stages of both strips once; loads rewrite only used rows
        for (int e = tid; e < 2 * S_ELEMS; e += NT) {
          lds[A_ELEMS + B_ELEMS + e] = T(0);
          lds[STAGE + A_ELEMS + B_ELEMS + e] = T(0);
        }
        __syncthreads();
      }
      la.load(A, g.lda, m0, g.M, k_lo, k_hi, tid);
      lb.load(B, g.ldb, n0, g.N, k_lo, k_hi, tid);
      if (cc) ls.load(Ac, g.ldac, rc0, nc_valid, k_lo, k_hi, tid);
      if (cr) lr.load(Br, g.ldbr, qc0, nq_valid, k_lo, k_hi, tid);
      la.store(lds, tid);
      lb.store(lds + A_ELEMS, tid);
      if (cc) ls.store(lds + A_ELEMS + B_ELEMS, nc, tid);
      if (cr) lr.store(lds + A_ELEMS + B_ELEMS + S_ELEMS, nq, tid);
      __syncthreads();
    }

    const int fr = lane & 15, fk = (lane >> 4) * FRAG;
    for (int kt = 0; kt < nk; ++kt) {
      const int cur = kt & 1;
      const bool more = kt + 1 < nk;
      if (more) {
        const int kn = k_lo + (kt + 1) * BK;
        la.load(A, g.lda, m0, g.M, kn, k_hi, tid);
        lb.load(B, g.ldb, n0, g.N, kn, k_hi, tid);
        if (cc) ls.load(Ac, g.ldac, rc0, nc_valid, kn, k_hi, tid);
        if (cr) lr.load(Br, g.ldbr, qc0, nq_valid, kn, k_hi, tid);
      }
      const T* sA = lds + cur * STAGE;
      const T* sB = sA + A_ELEMS;
      const T* sS = sB + B_ELEMS;
      const T* sR = sS + S_ELEMS;
#pragma unroll
      for (int kk = 0; kk < BK; kk += KI) {
        typename Mfma<T>::frag af[IM], bfr[JN];
#pragma unroll
        for (int i = 0; i < IM; ++i)
          af[i] = Mfma<T>::load(sA + (wm * WM + i * 16 + fr) * LDK + kk + fk);
#pragma unroll
        for (int j = 0; j < JN; ++j)
          bfr[j] = Mfma<T>::load(sB + (wn * WN + j * 16 + fr) * LDK + kk + fk);
#pragma unroll
        for (int i = 0; i < IM; ++i)
#pragma unroll
          for (int j = 0; j < JN; ++j) acc[i][j] = Mfma<T>::mma(af[i], bfr[j], acc[i][j]);
        if (PROT) {
          // wave-uniform branches keep every fragment index a compile-time
          // constant (a runtime index would send the arrays to scratch)
          if (cc) {
            const auto sf = Mfma<T>::load(sS + fr * LDK + kk + fk);
            if (wm == 0) {
#pragma unroll
              for (int j = 0; j < JS; ++j) accs[j] = Mfma<T>::mma(sf, bfr[j], accs[j]);
            } else {
#pragma unroll
              for (int j = 0; j < JS; ++j) accs[j] = Mfma<T>::mma(sf, bfr[JS + j], accs[j]);
            }
          }
          if (cr) {
            const auto rf = Mfma<T>::load(sR + fr * LDK + kk + fk);
            if (wn == 0) {
#pragma unroll
              for (int i = 0; i < IS; ++i) accr[i] = Mfma<T>::mma(rf, af[i], accr[i]);
            } else {
#pragma unroll
              for (int i = 0; i < IS; ++i) accr[i] = Mfma<T>::mma(rf, af[IS + i], accr[i]);
            }
          }
        }
      }
      if (more) {
        T* nA = lds + (cur ^ 1) * STAGE;
        la.store(nA, tid);
        lb.store(nA + A_ELEMS, tid);
        if (cc) ls.store(nA + A_ELEMS + B_ELEMS, nc, tid);
        if (cr) lr.store(nA + A_ELEMS + B_ELEMS + S_ELEMS, nq, tid);
      }
      __syncthreads();
    }

    // ---- epilogue: round to storage, inject faults ----
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int j = 0; j < JN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[i][j][r] = Storage<TC>::round(acc[i][j][r]);

    // A tile that an injected fault aims at takes the LDS path, where the
    // fault is written into the rounded tile before any verification.
    bool faulty = false;
    for (int f = 0; f < g.n_faults; ++f) {
      int fz, fm, fn;
      if (fault_target(g.map, g.N, g.faults[f], &fz, &fm, &fn) && fz == z && fm >= m0 &&
          fm < m0 + BM && fn >= n0 && fn < n0 + BN)
        faulty = true;
    }

    const int verify = PROT ? g.verify : 0;
    bool any = false;
    float* ccv = nullptr;
    float* rcv = nullptr;
    int* rowcnt = nullptr;
    int* colcnt = nullptr;
    const int nrb = BN / g.Rn > 0 ? BN / g.Rn : 1;   // row blocks per tile row
    const int ncb = BM / g.Rm;                       // column blocks per tile column
    if (PROT && (cc || cr)) {
      float* CsL = reinterpret_cast<float*>(smem);
      float* RsL = CsL + CSL;
      float* colp = RsL + RSL;
      float* rowp = colp + COLP;
      ccv = reinterpret_cast<float*>(smem + R0);
      rcv = ccv + CCV;
      rowcnt = reinterpret_cast<int*>(rcv + RCV);
      colcnt = rowcnt + BM * (BN / 16);

      // strip results to LDS
      if (cc) {
#pragma unroll
        for (int j = 0; j < JS; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            CsL[((lane >> 4) * 4 + r) * BN + wn * WN + (wm * JS + j) * 16 + fr] = accs[j][r];
      }
      if (cr) {
#pragma unroll
        for (int i = 0; i < IS; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            RsL[(wm * WM + (wn * IS + i) * 16 + fr) * 16 + (lane >> 4) * 4 + r] = accr[i][r];
      }
      // column partial sums per segment of min(Rm, WM) rows
      if (verify >= 1) {
        const int seg = g.Rm < WM ? g.Rm : WM;
#pragma unroll
        for (int j = 0; j < JN; ++j) {
          float s1 = 0.f, s2 = 0.f, sa = 0.f;
#pragma unroll
          for (int i = 0; i < IM; ++i) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int row = wm * WM + i * 16 + (lane >> 4) * 4 + r;
              const float v = acc[i][j][r];
              s1 += v;
              s2 += float((row & (g.Rm - 1)) + 1) * v;
              sa += is_finite(v) ? fabsf(v) : 0.f;
            }
            if (((i + 1) * 16) % seg == 0) {
              const float t1 = wsum16(s1), t2 = wsum16(s2), ta = wsum16(sa);
              const int c = (wm * WM + (i + 1) * 16 - seg) / 16;
              if (lane < 16) {
                float* p = colp + (c * BN + wn * WN + j * 16 + lane) * 3;
                p[0] = t1;
                p[1] = t2;
                p[2] = ta;
              }
              s1 = s2 = sa = 0.f;
            }
          }
        }
      }
      if (verify == 2) {
        const int seg = g.Rn < WN ? g.Rn : WN;
#pragma unroll
        for (int i = 0; i < IM; ++i) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row = wm * WM + i * 16 + (lane >> 4) * 4 + r;
            float s1 = 0.f, s2 = 0.f, sa = 0.f;
#pragma unroll
            for (int j = 0; j < JN; ++j) {
              const int col = wn * WN + j * 16 + fr;
              const float v = acc[i][j][r];
              s1 += v;
              s2 += float((col & (g.Rn - 1)) + 1) * v;
              sa += is_finite(v) ? fabsf(v) : 0.f;
              if (((j + 1) * 16) % seg == 0) {
                const float t1 = wsum_row(s1), t2 = wsum_row(s2), ta = wsum_row(sa);
                const int c = (wn * WN + (j + 1) * 16 - seg) / 16;
                if (fr == 0) {
                  float* p = rowp + (c * BM + row) * 3;
                  p[0] = t1;
                  p[1] = t2;
                  p[2] = ta;
                }
                s1 = s2 = sa = 0.f;
              }
            }
          }
        }
      }
      __syncthreads();
      // combine: propagated checksums (hi + lo) and detection per vector
      bool my_flag = false;
      if (cc) {
        const int segm = g.Rm < WM ? g.Rm : WM;
        for (int v = tid; v < ncb * BN; v += NT) {
          const int blk = v / BN, n = v % BN;
          float c1, c2;
          if constexpr (sizeof(T) == 2) {
            c1 = CsL[(2 * blk) * BN + n] + CsL[(nc + 2 * blk) * BN + n];
            c2 = CsL[(2 * blk + 1) * BN + n] + CsL[(nc + 2 * blk + 1) * BN + n];
          } else {
            c1 = CsL[(2 * blk) * BN + n];
            c2 = CsL[(2 * blk + 1) * BN + n];
          }
          ccv[v * 2] = c1;
          ccv[v * 2 + 1] = c2;
          if (verify >= 1 && m0 + blk * g.Rm < g.M && n0 + n < g.N && n0 + n >= g.verify_n_lo &&
              n0 + n < g.verify_n_hi) {
            float s1 = 0.f, sa = 0.f;
            for (int s = 0; s < g.Rm / segm; ++s) {
              const int c = (blk * g.Rm + s * segm) / 16;
              s1 += colp[(c * BN + n) * 3];
              sa += colp[(c * BN + n) * 3 + 2];
            }
            if (flagged(c1 - s1, sa, g.e_rel)) my_flag = true;
          }
        }
      }
      if (cr) {
        const int segn = g.Rn < WN ? g.Rn : WN;
        for (int u = tid; u < BM * nrb; u += NT) {
          const int row = u / nrb, rb = u % nrb;
          float c1, c2;
          if constexpr (sizeof(T) == 2) {
            c1 = RsL[row * 16 + 2 * rb] + RsL[row * 16 + nq + 2 * rb];
            c2 = RsL[row * 16 + 2 * rb + 1] + RsL[row * 16 + nq + 2 * rb + 1];
          } else {
            c1 = RsL[row * 16 + 2 * rb];
            c2 = RsL[row * 16 + 2 * rb + 1];
          }
          rcv[u * 2] = c1;
          rcv[u * 2 + 1] = c2;
          if (verify == 2 && m0 + row < g.M && n0 + rb * g.Rn < g.N) {
            float s1 = 0.f, sa = 0.f;
            for (int s = 0; s < g.Rn / segn; ++s) {
              const int c = (rb * g.Rn + s * segn) / 16;
              s1 += rowp[(c * BM + row) * 3];
              sa += rowp[(c * BM + row) * 3 + 2];
            }
            if (flagged(c1 - s1, sa, g.e_rel)) my_flag = true;
          }
        }
      }
      any = __syncthreads_or(my_flag);
    }

    if (!any && !faulty) {
      // fast path: store straight from registers
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int j = 0; j < JN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = m0 + wm * WM + i * 16 + (lane >> 4) * 4 + r;
            const int n = n0 + wn * WN + j * 16 + fr;
            if (m < g.M && n < g.N) C[int64_t(m) * g.ldc + n] = Storage<TC>::store(acc[i][j][r]);
          }
    } else {
      TC* tile = reinterpret_cast<TC*>(smem);  // overlays dead partial sums / operand stages
      __syncthreads();
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int j = 0; j < JN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            tile[(wm * WM + i * 16 + (lane >> 4) * 4 + r) * BN + wn * WN + j * 16 + fr] =
                Storage<TC>::store(acc[i][j][r]);
      slow_path(g, tile, A, B, C, z, m0, n0, k_lo, k_hi, ccv, rcv, rowcnt, colcnt, nrb, ncb,
                cc ? verify : 0, tid);
    }

    // propagated checksums for the consumers downstream
    if (PROT && cc && g.Cc != nullptr) {
      float* Cc = g.Cc + b0 * g.sCc0 + b1 * g.sCc1;
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
  }

  // Slow path: the tile goes to LDS and EEC-ABFT runs there (one thread per
  // vector, as in the paper's Fig. 4), then the tile is stored.
  __device__ static __forceinline__ void slow_path(
      const GemmDesc& g, TC* tile, const T* A, const T* B, TC* C, int z, int m0, int n0,
      int k_lo, int k_hi, float* ccv, float* rcv, int* rowcnt, int* colcnt, int nrb, int ncb,
      int verify, int tid) {
    // injected faults (test-only), after rounding to storage
    if (tid == 0) {
      for (int f = 0; f < g.n_faults; ++f) {
        const abft_fault ft = g.faults[f];
        int fz, fm, fn;
        if (fault_target(g.map, g.N, ft, &fz, &fm, &fn) && fz == z && fm >= m0 &&
            fm < m0 + BM && fn >= n0 && fn < n0 + BN)
          tile[(fm - m0) * BN + fn - n0] = Storage<TC>::store(Storage<TC>::round(ft.value));
      }
    }
    if (verify >= 1)
      for (int e = tid; e < BM * (BN / 16) + (BM / 16) * BN; e += NT) rowcnt[e] = 0;
    __syncthreads();
    if (verify >= 1) passes(g, tile, A, B, z, m0, n0, k_lo, k_hi, ccv, rcv, rowcnt, colcnt, nrb,
                            ncb, verify, tid);
    for (int e = tid; e < BM * BN; e += NT) {
      const int row = e / BN, col = e % BN;
      if (m0 + row < g.M && n0 + col < g.N) C[int64_t(m0 + row) * g.ldc + n0 + col] = tile[e];
    }
  }

  // EEC-ABFT on the LDS tile, one thread per vector (as in the paper's Fig. 4).
  __device__ static __forceinline__ void passes(
      const GemmDesc& g, TC* tile, const T* A, const T* B, int z, int m0, int n0, int k_lo,
      int k_hi, float* ccv, float* rcv, int* rowcnt, int* colcnt, int nrb, int ncb, int verify,
      int tid) {

    const int Rm = g.Rm, Rn = g.Rn;
    auto in_col = [&](int blk, int n) {
      return m0 + blk * Rm < g.M && n0 + n < g.N && n0 + n >= g.verify_n_lo &&
             n0 + n < g.verify_n_hi;
    };
    auto in_row = [&](int row, int rb) { return m0 + row < g.M && n0 + rb * Rn < g.N; };
    auto correct = [&](int lr, int lc, const TC* vec, int stride, int nvec, int idx, float c1,
                       float d1) {
      const float old = Storage<TC>::load(tile[lr * BN + lc]);
      int action;
      float val;
      if (g.recompute) {
        val = recompute_elem<T, TC, AK, BKM>(g, A, B, m0 + lr, n0 + lc, k_lo, k_hi);
        action = ABFT_ACT_RECOMPUTE;
      } else {
        val = fix_by_checksum<TC>(vec, stride, nvec, idx, c1, d1, g.tc, &action);
      }
      tile[lr * BN + lc] = Storage<TC>::store(val);
      const EvCoord ec = map_coord(g.map, z, m0 + lr, n0 + lc);
      record_event(g.report, ec.op, ec.b, ec.h, ec.row, ec.col, classify(old, g.tn), action, old);
    };

    // 1. column pass
    for (int v = tid; v < ncb * BN; v += NT) {
      const int blk = v / BN, n = v % BN;
      if (!in_col(blk, n)) continue;
      const TC* vec = tile + blk * Rm * BN + n;
      const EecResult res = eec_locate<TC>(vec, BN, Rm, ccv[v * 2], ccv[v * 2 + 1], g.e_rel, g.tn);
      if (res.status == EEC_LOCATED) {
        const int lr = blk * Rm + res.index;
        correct(lr, n, vec, BN, Rm, res.index, ccv[v * 2], res.d1);
        if (verify == 2) atomicAdd(&rowcnt[lr * nrb + n / Rn], 1);
      }
    }
    __syncthreads();
    if (verify == 2) {
      // 2a. refresh row checksums of row vectors with >= 2 corrections (1R)
      for (int u = tid; u < BM * nrb; u += NT) {
        const int row = u / nrb, rb = u % nrb;
        if (in_row(row, rb) && rowcnt[u] >= 2)
          vec_checksums<TC>(tile + row * BN + rb * Rn, 1, Rn, &rcv[u * 2], &rcv[u * 2 + 1]);
      }
      __syncthreads();
      // 2b. row pass
      for (int u = tid; u < BM * nrb; u += NT) {
        const int row = u / nrb, rb = u % nrb;
        if (!in_row(row, rb)) continue;
        const TC* vec = tile + row * BN + rb * Rn;
        const EecResult res = eec_locate<TC>(vec, 1, Rn, rcv[u * 2], rcv[u * 2 + 1], g.e_rel, g.tn);
        if (res.status == EEC_LOCATED) {
          const int lc = rb * Rn + res.index;
          correct(row, lc, vec, 1, Rn, res.index, rcv[u * 2], res.d1);
          atomicAdd(&colcnt[(row / Rm) * BN + lc], 1);
        }
      }
      __syncthreads();
      // 2c. refresh column checksums of column vectors with >= 2 corrections (1C)
      for (int v = tid; v < ncb * BN; v += NT) {
        const int blk = v / BN, n = v % BN;
        if (in_col(blk, n) && colcnt[v] >= 2)
          vec_checksums<TC>(tile + blk * Rm * BN + n, BN, Rm, &ccv[v * 2], &ccv[v * 2 + 1]);
      }
      __syncthreads();
    }
    // 3. final check: anything still inconsistent is uncorrectable (2-D)
    for (int v = tid; v < ncb * BN; v += NT) {
      const int blk = v / BN, n = v % BN;
      if (!in_col(blk, n)) continue;
      if (vec_flagged<TC>(tile + blk * Rm * BN + n, BN, Rm, ccv[v * 2], g.e_rel)) {
        const EvCoord ec = map_coord(g.map, z, m0 + blk * Rm, n0 + n);
        record_event(g.report, ec.op, ec.b, ec.h, ec.row, ec.col, ABFT_KIND_NONE,
                     ABFT_ACT_UNCORRECTABLE, 0.f);
      }
    }
    if (verify == 2) {
      for (int u = tid; u < BM * nrb; u += NT) {
        const int row = u / nrb, rb = u % nrb;
        if (!in_row(row, rb)) continue;
        if (vec_flagged<TC>(tile + row * BN + rb * Rn, 1, Rn, rcv[u * 2], g.e_rel)) {
          const EvCoord ec = map_coord(g.map, z, m0 + row, n0 + rb * Rn);
          record_event(g.report, ec.op, ec.b, ec.h, ec.row, ec.col, ABFT_KIND_NONE,
                       ABFT_ACT_UNCORRECTABLE, 0.f);
        }
      }
    }
    __syncthreads();
  }
};

template <class T, class TC, bool AK, bool BKM, int BM, int BN, bool PROT>
__global__ __launch_bounds__(NT) void gemm_kernel(GemmDesc g) {
  extern __shared__ __align__(16) char smem[];
  Gemm<T, TC, AK, BKM, BM, BN, PROT>::run(g, smem);
}

template <class T, class TC, bool AK, bool BKM, int BM, int BN, bool PROT>
hipError_t launch_t(const GemmDesc& g, hipStream_t s) {
  using G = Gemm<T, TC, AK, BKM, BM, BN, PROT>;
  auto kern = gemm_kernel<T, TC, AK, BKM, BM, BN, PROT>;
  const size_t lds = G::LDS_BYTES;
  if (lds > 160 * 1024) return hipErrorInvalidValue;  // this tile does not fit gfx950 LDS
  static bool attr_set = false;  // per instantiation; harmless if repeated
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  dim3 grid(tiles, g.nb0 * g.nb1);
  if (tiles == 0 || g.nb0 * g.nb1 == 0) return hipSuccess;
  hipLaunchKernelGGL(kern, grid, dim3(NT), lds, s, g);
  return hipGetLastError();
}

template <class T, class TC, bool AK, bool BKM, bool PROT>
hipError_t launch_tile(const GemmDesc& g, Tile tile, hipStream_t s) {
  switch (tile) {
    case Tile::T256x128: return launch_t<T, TC, AK, BKM, 256, 128, PROT>(g, s);
    case Tile::T128x128: return launch_t<T, TC, AK, BKM, 128, 128, PROT>(g, s);
    case Tile::T128x64: return launch_t<T, TC, AK, BKM, 128, 64, PROT>(g, s);
  }
  return hipErrorInvalidValue;
}

template <class T, class TC, bool PROT>
hipError_t launch_layout(const GemmDesc& g, Layout la, Layout lb, Tile tile, hipStream_t s) {
  const bool ak = la == Layout::KMajor, bk = lb == Layout::KMajor;
  if (ak && !bk) return launch_tile<T, TC, true, false, PROT>(g, tile, s);
  if (ak && bk) return launch_tile<T, TC, true, true, PROT>(g, tile, s);
  if (!ak && !bk) return launch_tile<T, TC, false, false, PROT>(g, tile, s);
  return hipErrorInvalidValue;  // (MN-major A, K-major B) is not used by the layer
}

}  // namespace

hipError_t launch_gemm(const GemmDesc& g, int dtype, bool c_fp32, Layout la, Layout lb,
                       Tile tile, hipStream_t stream) {
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
