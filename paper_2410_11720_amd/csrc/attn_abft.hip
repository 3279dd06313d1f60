// Host orchestration of the ABFT-protected attention layer and the C ABI
// (include/attn_abft.h).
//
// Forward, per the protection sections of paper Sec. 4.4:
//   encode  W^V row checksums per head; X column checksums per R-token
//           block and row checksums per head block (the latter for dW)
//   S_AS    [Q|K|V] = X Wqkv with Q^c|K^c|V^c = X^c Wqkv as extra MFMA rows
//           and V^r = X W^V r as extra MFMA columns on the V tiles; root
//           check of Q, K, V (column pass, corrected by recompute)
//           AS = Q K^T per head, AS^c = Q^c K^T, AS^r = Q (K^c)^T, two-sided
//           verification (Sec. 4.3)
//   softmax AP with column checksums AP^c (and row checksums for dV)
//   S_CL    CL = AP V per head, CL^c = AP^c V, CL^r = AP V^r, two-sided
//   S_O     O = CL Wo, O^c = CL^c Wo, column pass
// Backward (extension): every GEMM output carries a propagated column
// checksum and gets a column pass; see attn_abft_backward below.
#include <cmath>
#include <cstring>
#include <mutex>

#include "abft_internal.hpp"

namespace abft {

float stored_threshold(float t, int dtype) {
  if (dtype == ABFT_FP32) return t;
  uint32_t u;
  std::memcpy(&u, &t, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return t;
  u += 0x7fffu + ((u >> 16) & 1u);
  u &= 0xffff0000u;
  float r;
  std::memcpy(&r, &u, 4);
  return r;
}

namespace {

constexpr size_t ALIGN = 256;
size_t align_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

struct Dims {
  int64_t B, S, H, nh, d, R, nq, T;
  size_t es;
};

struct Layout_ {
  size_t qkv, ap, cl, as, das, dcl, dqkv;
  size_t xc, xr, wvr, qkvc, vr, apc, apr, clc, clr, doc, dclc, dasc, dasr, dqkvc;
  // bf16 images of X^c, dO^c and dQKV^c (four rows per block): the GEMMs
  // that take them as column strips copy them like operand tiles
  size_t xci, doci, dqkvci;
  size_t xri;  // bf16 image of X^r, transposed ([nh][4][T]): dW^QKV's strip
  size_t clri; // the same of CL^r, written by the fused forward: dW^O's strip
  size_t wvri; // the same of W^V r ([nh][4][H]): the QKV GEMM's row strip
  size_t clci; // bf16 image of CL^c (fused form): the output projection's strip
  size_t skp, skc;  // split-K partials of the weight gradients and their checksums
  size_t stats;     // fused forward: softmax max and sum per query [B][nh][S][2]
  size_t drow;      // fused backward: D = dCL . CL per query [B][nh][S]
  size_t total;
};

// K slices for a weight-gradient GEMM (M x N tiles of 128 x 128, long K):
// enough slices to give at least 256 workgroups, each slice at least 256
// deep.
int splitk_for(int64_t M, int64_t N, int64_t K, bool prot) {
  const int64_t tiles = ((M + 127) / 128) * ((N + 127) / 128);
  int ks = 1;
  // smallest power of two that fills every CU once (fewer slices, less
  // partial-sum traffic), with K slices of at least 256; a checked tile in
  // one slice stages its fp32 tile for the column check in an epilogue
  // area that still leaves two workgroups per CU
  (void)prot;
  while (tiles * ks < 256 && K / (2 * ks) >= 256 && ks < 16) ks *= 2;
  return ks;
}

bool make_dims(const attn_abft_config* c, Dims* d) {
  if (!c || c->batch < 1 || c->seq < 1 || c->hidden < 1 || c->heads < 1) return false;
  if (c->hidden % c->heads) return false;
  d->B = c->batch;
  d->S = c->seq;
  d->H = c->hidden;
  d->nh = c->heads;
  d->d = c->hidden / c->heads;
  d->R = c->block_rows;
  if (d->R < 1 || d->S % d->R) return false;
  d->nq = d->S / d->R;
  d->T = d->B * d->S;
  d->es = c->dtype == ABFT_FP32 ? 4 : 2;
  return true;
}

Layout_ make_layout(const Dims& d) {
  Layout_ L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  const size_t SS = size_t(d.B) * d.nh * d.S * d.S;
  L.qkv = take(size_t(d.T) * 3 * d.H * d.es);
  L.ap = take(SS * d.es);
  L.cl = take(size_t(d.T) * d.H * d.es);
  L.as = take(SS * d.es);
  L.das = take(SS * d.es);
  L.dcl = take(size_t(d.T) * d.H * d.es);
  L.dqkv = take(size_t(d.T) * 3 * d.H * d.es);
  const size_t f = 4;
  L.xc = take(size_t(d.B) * d.nq * 2 * d.H * f);
  L.xr = take(size_t(d.T) * d.nh * 2 * f);
  L.wvr = take(size_t(d.H) * d.nh * 2 * f);
  L.qkvc = take(size_t(d.B) * d.nq * 2 * 3 * d.H * f);
  L.vr = take(size_t(d.T) * d.nh * 2 * f);
  L.apc = take(size_t(d.B) * d.nh * d.nq * 2 * d.S * f);
  L.apr = take(size_t(d.B) * d.nh * d.S * d.nq * 2 * f);
  L.clc = take(size_t(d.B) * d.nq * 2 * d.H * f);
  L.clr = take(size_t(d.T) * d.nh * 2 * f);
  L.doc = take(size_t(d.B) * d.nq * 2 * d.H * f);
  L.dclc = take(size_t(d.B) * d.nq * 2 * d.H * f);
  L.dasc = take(size_t(d.B) * d.nh * d.nq * 2 * d.S * f);
  L.dasr = take(size_t(d.B) * d.nh * d.S * d.nq * 2 * f);
  L.dqkvc = take(size_t(d.B) * d.nq * 2 * 3 * d.H * f);
  L.xci = take(size_t(d.B) * d.nq * 4 * d.H * 2);
  L.wvri = take(size_t(d.nh) * 4 * d.H * 2);
  L.clci = take(size_t(d.B) * d.nq * 4 * d.H * 2);
  L.doci = take(size_t(d.B) * d.nq * 4 * d.H * 2);
  L.dqkvci = take(size_t(d.B) * d.nq * 4 * 3 * d.H * 2);
  L.xri = take(size_t(d.nh) * 4 * d.T * 2);
  const int ks1 = splitk_for(d.H, 3 * d.H, d.T, true), ks2 = splitk_for(d.H, d.H, d.T, true);
  const size_t p1 = ks1 > 1 ? size_t(ks1) * d.H * 3 * d.H : 0;
  const size_t p2 = ks2 > 1 ? size_t(ks2) * d.H * d.H : 0;
  const size_t c1 = ks1 > 1 ? size_t(ks1) * 2 * d.nh * 3 * d.H : 0;
  const size_t c2 = ks2 > 1 ? size_t(ks2) * 2 * d.nh * d.H : 0;
  L.skp = take((p1 > p2 ? p1 : p2) * f);
  L.skc = take((c1 > c2 ? c1 : c2) * f);
  L.total = off;
  return L;
}

// Forward-only layout of the fused form (what attn_abft_forward with
// ABFT_FLAG_FUSED writes and reads when no backward follows): projections,
// context, the checksums the fused kernel and the output projection take,
// and the softmax statistics. Offsets of tensors outside it stay 0 and are
// never used on that path.
Layout_ make_layout_fused_forward(const Dims& d) {
  Layout_ L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  const size_t f = 4;
  L.qkv = take(size_t(d.T) * 3 * d.H * d.es);
  L.cl = take(size_t(d.T) * d.H * d.es);
  L.xc = take(size_t(d.B) * d.nq * 2 * d.H * f);
  L.wvr = take(size_t(d.H) * d.nh * 2 * f);
  L.qkvc = take(size_t(d.B) * d.nq * 2 * 3 * d.H * f);
  L.vr = take(size_t(d.T) * d.nh * 2 * f);
  L.clc = take(size_t(d.B) * d.nq * 2 * d.H * f);
  L.clr = take(size_t(d.T) * d.nh * 2 * f);
  L.stats = take(size_t(d.B) * d.nh * d.S * 2 * f);
  L.xci = take(size_t(d.B) * d.nq * 4 * d.H * 2);
  L.wvri = take(size_t(d.nh) * 4 * d.H * 2);
  L.clci = take(size_t(d.B) * d.nq * 4 * d.H * 2);
  L.clri = take(size_t(d.nh) * 4 * d.T * 2);
  L.total = off;
  return L;
}

// Layout of the fused form with a backward: no score-shaped tensor (AS,
// AP, dAS and their checksums); the fused backward core's row checksums
// and row terms instead. Offsets of tensors outside it stay 0 and are
// never used on the fused path.
Layout_ make_layout_fused(const Dims& d) {
  Layout_ L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  const size_t f = 4;
  L.qkv = take(size_t(d.T) * 3 * d.H * d.es);
  L.cl = take(size_t(d.T) * d.H * d.es);
  L.dcl = take(size_t(d.T) * d.H * d.es);
  L.dqkv = take(size_t(d.T) * 3 * d.H * d.es);
  L.xc = take(size_t(d.B) * d.nq * 2 * d.H * f);
  L.xr = take(size_t(d.T) * d.nh * 2 * f);
  L.wvr = take(size_t(d.H) * d.nh * 2 * f);
  L.qkvc = take(size_t(d.B) * d.nq * 2 * 3 * d.H * f);
  L.vr = take(size_t(d.T) * d.nh * 2 * f);
  L.clc = take(size_t(d.B) * d.nq * 2 * d.H * f);
  L.clr = take(size_t(d.T) * d.nh * 2 * f);
  L.doc = take(size_t(d.B) * d.nq * 2 * d.H * f);
  L.dclc = take(size_t(d.B) * d.nq * 2 * d.H * f);
  L.dqkvc = take(size_t(d.B) * d.nq * 2 * 3 * d.H * f);
  L.xci = take(size_t(d.B) * d.nq * 4 * d.H * 2);
  L.wvri = take(size_t(d.nh) * 4 * d.H * 2);
  L.clci = take(size_t(d.B) * d.nq * 4 * d.H * 2);
  L.doci = take(size_t(d.B) * d.nq * 4 * d.H * 2);
  L.dqkvci = take(size_t(d.B) * d.nq * 4 * 3 * d.H * 2);
  L.xri = take(size_t(d.nh) * 4 * d.T * 2);
  const int ks1 = splitk_for(d.H, 3 * d.H, d.T, true), ks2 = splitk_for(d.H, d.H, d.T, true);
  const size_t p1 = ks1 > 1 ? size_t(ks1) * d.H * 3 * d.H : 0;
  const size_t p2 = ks2 > 1 ? size_t(ks2) * d.H * d.H : 0;
  const size_t c1 = ks1 > 1 ? size_t(ks1) * 2 * d.nh * 3 * d.H : 0;
  const size_t c2 = ks2 > 1 ? size_t(ks2) * 2 * d.nh * d.H : 0;
  L.skp = take((p1 > p2 ? p1 : p2) * f);
  L.skc = take((c1 > c2 ? c1 : c2) * f);
  L.stats = take(size_t(d.B) * d.nh * d.S * 2 * f);
  L.drow = take(size_t(d.B) * d.nh * d.S * f);
  L.clri = take(size_t(d.nh) * 4 * d.T * 2);
  L.total = off;
  return L;
}

Layout_ layout_for(const attn_abft_config* c, const Dims& d) {
  return (c->flags & ABFT_FLAG_FUSED) ? make_layout_fused(d) : make_layout(d);
}

int validate(const attn_abft_config* c, Dims* d) {
  if (!make_dims(c, d)) return ABFT_ERR_INVALID;
  if (c->dtype != ABFT_BF16 && c->dtype != ABFT_FP32) return ABFT_ERR_UNSUPPORTED;
  if (c->causal != 0 && c->causal != 1) return ABFT_ERR_INVALID;
  const int64_t R = d->R;
  if ((R & (R - 1)) != 0 || R > 128 || R < (c->dtype == ABFT_FP32 ? 16 : 32))
    return ABFT_ERR_UNSUPPORTED;
  if (d->d != 64 && d->d != 128) return ABFT_ERR_UNSUPPORTED;
  if (d->S % 8 || d->H % 8) return ABFT_ERR_UNSUPPORTED;
  if (d->S > 4096) return ABFT_ERR_UNSUPPORTED;  // softmax keeps a row in registers
  if ((c->flags & ABFT_FLAG_FUSED) && (c->dtype != ABFT_BF16 || d->S % 128))
    return ABFT_ERR_UNSUPPORTED;
  if (!(c->t_near_inf >= 0.f) || !(c->t_correct >= 0.f) || !(c->e_rel >= 0.f))
    return ABFT_ERR_INVALID;
  return ABFT_OK;
}

int check_device() {
  static std::mutex mu;
  static int cached[64];
  static bool init[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ABFT_ERR_HIP;
  if (dev < 0 || dev >= 64) return ABFT_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(mu);
  if (!init[dev]) {
    hipDeviceProp_t p;
    if (hipGetDeviceProperties(&p, dev) != hipSuccess) return ABFT_ERR_HIP;
    cached[dev] = std::strncmp(p.gcnArchName, "gfx950", 6) == 0 ? ABFT_OK : ABFT_ERR_UNSUPPORTED;
    init[dev] = true;
  }
  return cached[dev];
}

struct Params {
  float e_rel, tn, tc, scale;
  bool prot, root, sec_as, sec_cl, sec_o, sec_bwd;
};

Params make_params(const attn_abft_config* c, const Dims& d) {
  Params p;
  p.e_rel = c->e_rel > 0.f ? c->e_rel : (c->dtype == ABFT_FP32 ? std::ldexp(1.f, -13)
                                                                : std::ldexp(1.f, -4));
  p.tn = stored_threshold(c->t_near_inf > 0.f ? c->t_near_inf : 1e10f, c->dtype);
  p.tc = c->t_correct > 0.f ? c->t_correct : 1e5f;
  p.scale = c->scale > 0.f ? c->scale : 1.f / std::sqrt(float(d.d));
  p.prot = !(c->flags & ABFT_FLAG_UNPROTECTED);
  p.root = (c->flags & ABFT_FLAG_ROOT_CHECK) != 0;
  p.sec_as = p.prot && (c->sections & ABFT_SEC_AS);
  p.sec_cl = p.prot && (c->sections & ABFT_SEC_CL);
  p.sec_o = p.prot && (c->sections & ABFT_SEC_O);
  p.sec_bwd = p.prot && (c->sections & ABFT_SEC_BWD);
  return p;
}

// Projection tile: 128 x 128 (two workgroups per CU with the direct
// operand path); a 256 x 128 tile fits one per CU and measured slower.
Tile proj_tile() { return Tile::T128x128; }

#define CK(x)                                          \
  do {                                                 \
    hipError_t e_ = (x);                               \
    if (e_ != hipSuccess) return ABFT_ERR_HIP;         \
  } while (0)

// The launch descriptor of a weight-gradient GEMM (MN-major operands, fp32
// output) split over K into ks partials when that fills the GPU better
// (the GEMM itself when ks is 1).
GemmDesc wgrad_slices(const GemmDesc& g, float* part, float* part_c, int* ks_out) {
  const int ks = splitk_for(g.M, g.N, g.K, g.Ac != nullptr || g.Br != nullptr || g.verify != 0);
  *ks_out = ks;
  if (ks <= 1) return g;
  GemmDesc sg = g;
  sg.splitk = ks;
  sg.C = part;
  sg.ldc = g.N;
  sg.sCk = int64_t(g.M) * g.N;
  sg.Cc = g.Ac != nullptr ? part_c : nullptr;
  sg.ldcc = g.N;
  sg.sCck = int64_t(2 * (g.M / g.Rm)) * g.N;
  sg.n_faults = 0;
  sg.faults = nullptr;
  return sg;
}

// A weight-gradient GEMM: its slices, then (split) the reduction that sums
// and verifies them.
hipError_t launch_wgrad(const GemmDesc& g, int dt, float* part, float* part_c, hipStream_t s) {
  int ks = 1;
  const GemmDesc sg = wgrad_slices(g, part, part_c, &ks);
  hipError_t e = launch_gemm(sg, dt, true, Layout::MNMajor, Layout::MNMajor, Tile::T128x128, s);
  if (e != hipSuccess || ks <= 1) return e;
  GemmDesc rg = g;
  rg.splitk = ks;
  return launch_splitk_reduce(rg, part, part_c, dt, Layout::MNMajor, Layout::MNMajor, s);
}

// A weight gradient w and an independent projection pj (K-major operands;
// either may be absent): in one launch when they qualify, so that each
// fills the CUs the other leaves idle in its last round; else pj, then w.
hipError_t wgrad_with_proj(const GemmDesc* w, const GemmDesc* pj, int dt, float* part,
                           float* part_c, hipStream_t s) {
  if (w && pj) {
    int ks = 1;
    const GemmDesc sg = wgrad_slices(*w, part, part_c, &ks);
    const hipError_t e = launch_gemm_pair(sg, *pj, dt, s);
    if (e == hipSuccess) {
      if (ks <= 1) return hipSuccess;
      GemmDesc rg = *w;
      rg.splitk = ks;
      return launch_splitk_reduce(rg, part, part_c, dt, Layout::MNMajor, Layout::MNMajor, s);
    }
    if (e != hipErrorNotSupported) return e;
  }
  if (pj) {
    const hipError_t e = launch_gemm(*pj, dt, false, Layout::KMajor, Layout::KMajor, proj_tile(), s);
    if (e != hipSuccess) return e;
  }
  return w ? launch_wgrad(*w, dt, part, part_c, s) : hipSuccess;
}

GemmDesc base_desc(const Params& p, const abft_fault* faults, int n_faults, abft_report* rep) {
  GemmDesc g;
  g.e_rel = p.e_rel;
  g.tn = p.tn;
  g.tc = p.tc;
  g.recompute = p.root ? 1 : 0;
  g.faults = faults;
  g.n_faults = n_faults;
  g.report = rep;
  return g;
}

}  // namespace
}  // namespace abft

using namespace abft;

extern "C" {

size_t attn_abft_workspace_bytes(const attn_abft_config* cfg) {
  Dims d;
  if (validate(cfg, &d) != ABFT_OK) return 0;
  return layout_for(cfg, d).total;
}

size_t attn_abft_report_bytes(int32_t capacity) {
  if (capacity < 0) return 0;
  return sizeof(abft_report) + size_t(capacity) * sizeof(abft_event);
}

int attn_abft_report_init(abft_report* report, int32_t capacity, void* stream) {
  if (!report || capacity < 0) return ABFT_ERR_INVALID;
  CK(launch_report_reset(report, capacity, true, static_cast<hipStream_t>(stream)));
  return ABFT_OK;
}

int attn_abft_workspace_offsets(const attn_abft_config* cfg, size_t* qkv_offset,
                                size_t* ap_offset, size_t* cl_offset) {
  Dims d;
  if (validate(cfg, &d) != ABFT_OK) return ABFT_ERR_INVALID;
  if ((cfg->flags & ABFT_FLAG_FUSED) && ap_offset) return ABFT_ERR_UNSUPPORTED;  // no AP kept
  const Layout_ L = layout_for(cfg, d);
  if (qkv_offset) *qkv_offset = L.qkv;
  if (ap_offset) *ap_offset = L.ap;
  if (cl_offset) *cl_offset = L.cl;
  return ABFT_OK;
}

int attn_abft_workspace_tensor(const attn_abft_config* cfg, int32_t which, size_t* offset) {
  Dims d;
  if (validate(cfg, &d) != ABFT_OK || !offset) return ABFT_ERR_INVALID;
  const Layout_ L = layout_for(cfg, d);
  // the fused form keeps no score-shaped tensor
  if ((cfg->flags & ABFT_FLAG_FUSED) && (which == 1 || which == 2 || which >= 6))
    return which <= 8 ? ABFT_ERR_UNSUPPORTED : ABFT_ERR_INVALID;
  switch (which) {
    case 0: *offset = L.qkv; return ABFT_OK;
    case 1: *offset = L.as; return ABFT_OK;
    case 2: *offset = L.ap; return ABFT_OK;
    case 3: *offset = L.cl; return ABFT_OK;
    case 4: *offset = L.dqkv; return ABFT_OK;
    case 5: *offset = L.dcl; return ABFT_OK;
    case 6: *offset = L.apc; return ABFT_OK;
    case 7: *offset = L.apr; return ABFT_OK;
    case 8: *offset = L.das; return ABFT_OK;
  }
  return ABFT_ERR_INVALID;
}

}  // extern "C"

namespace abft {
namespace {

// The forward chain over a workspace at ws laid out by L (arguments
// already validated).
int forward_impl(const attn_abft_config* cfg, const Dims& d, const Layout_& L, const Params& p,
                 const void* X, const void* Wqkv, const void* Wo, void* O, char* ws,
                 const abft_fault* faults, int32_t n_faults, abft_report* report,
                 uint32_t stages, hipStream_t s) {
  const int dt = cfg->dtype;
  auto F = [&](size_t off) { return reinterpret_cast<float*>(ws + off); };
  const char* Xc = static_cast<const char*>(X);
  const char* Wc = static_cast<const char*>(Wqkv);
  const int64_t B = d.B, S = d.S, H = d.H, nh = d.nh, hd = d.d, R = d.R, nq = d.nq, T = d.T;
  const size_t es = d.es;

  // Checksum operands, each computed when any enabled section consumes it
  // (the backward's propagated checksums come from the forward: X^r for dW,
  // AP^r for dV, CL^r for dWo; a forward that precedes a protected backward
  // must have ABFT_SEC_BWD set).
  const bool fused = (cfg->flags & ABFT_FLAG_FUSED) != 0;
  // Q^c, K^c; the V root check (the fused form verifies V in every mode);
  // Q^c, K^c and V^c for a fused backward's checks
  const bool need_xc = p.sec_as || ((p.root || fused) && p.sec_cl) || (fused && p.sec_bwd);
  const bool need_vr = p.sec_cl || p.sec_bwd;             // V^r -> CL^r
  const bool need_apc = p.sec_cl || p.sec_o;              // AP^c -> CL^c -> O^c
  // encode (Sec. 4.6): W^V row checksums per head; X column and row
  // checksums; the report is cleared in the same launch
  {
    EncodeJob jobs[2];
    int nj = 0;
    if ((stages & ABFT_STAGE_ENCODE) && need_vr) {
      EncodeJob& e = jobs[nj++];
      e.A = Wc + 2 * H * es; e.batch = 1; e.rows = H; e.cols = H; e.ld = 3 * H;
      // row checksums only: any row block; 128 rows fill a workgroup's loads
      e.Rb = H % 128 == 0 ? 128 : (H % 64 == 0 ? 64 : 32);
      e.Cb = int(hd); e.row_chk = F(L.wvr);
      if (es == 2) { e.row_img = reinterpret_cast<uint16_t*>(ws + L.wvri); e.ldri = H; }
    }
    if ((stages & ABFT_STAGE_ENCODE) && (need_xc || p.sec_bwd)) {
      EncodeJob& e = jobs[nj++];
      e.A = X; e.batch = B; e.rows = S; e.cols = H; e.ld = H; e.batch_stride = S * H;
      e.Rb = int(R); e.Cb = int(hd);
      e.col_chk = need_xc ? F(L.xc) : nullptr;
      e.row_chk = p.sec_bwd ? F(L.xr) : nullptr;
      if (p.sec_bwd && es == 2) {
        e.row_img = reinterpret_cast<uint16_t*>(ws + L.xri);
        e.ldri = T;
      }
      if (need_xc && es == 2) {
        e.col_img = reinterpret_cast<uint16_t*>(ws + L.xci);
        e.ldci = H;
      }
    }
    CK(launch_encode_jobs(jobs, nj, dt,
                          (cfg->flags & ABFT_FLAG_REPORT_APPEND) ? nullptr : report, s));
  }

  // [Q|K|V] = X Wqkv
  if (stages & ABFT_STAGE_QKV) {
    GemmDesc g = base_desc(p, faults, n_faults, report);
    g.M = int(T); g.N = int(3 * H); g.K = int(H);
    g.A = X; g.lda = H;
    g.B = Wqkv; g.ldb = 3 * H;
    g.C = ws + L.qkv; g.ldc = 3 * H;
    if (need_xc) {
      g.Ac = F(L.xc); g.ldac = H; g.Rm = int(R);
      g.Cc = F(L.qkvc); g.ldcc = 3 * H;
      if (es == 2) { g.Aci = reinterpret_cast<const uint16_t*>(ws + L.xci); g.ldaci = H; }
    }
    if (need_vr) {
      g.Br = F(L.wvr); g.ldbr = 2 * nh; g.Rn = int(hd); g.cr_n_begin = int(2 * H);
      if (es == 2) { g.Bri = reinterpret_cast<const uint16_t*>(ws + L.wvri); g.ldbri = H; }
      g.Cr = F(L.vr); g.ldcr = 2 * nh;
    }
    // the fused form's score checks have one side per pass, which cannot
    // see an error of the operand on that side (it moves a score row or
    // column together with its checksums): it verifies Q, K and V here in
    // every mode, fixed from their checksums without the root check
    if ((p.root || fused) && (p.sec_as || p.sec_cl)) {
      g.verify = 1;
      g.verify_n_lo = p.sec_as ? 0 : int(2 * H);
      g.verify_n_hi = p.sec_cl ? int(3 * H) : int(2 * H);
    }
    g.map.op_base = ABFT_OP_Q; g.map.op_span = int(H); g.map.rows_per_b = int(S);
    g.map.head_cols = int(hd);
    CK(launch_gemm(g, dt, false, Layout::KMajor, Layout::MNMajor, proj_tile(), s));
  }
  if (fused && (stages & (ABFT_STAGE_SCORE | ABFT_STAGE_SOFTMAX | ABFT_STAGE_CONTEXT))) {
    // score, softmax and context in one kernel (no AS or AP in memory)
    FusedDesc fd;
    fd.B = int(B); fd.nh = int(nh); fd.S = int(S); fd.H = int(H); fd.D = int(hd); fd.R = int(R);
    fd.causal = cfg->causal;
    fd.scale = p.scale;
    fd.qkv = ws + L.qkv;
    fd.qkvc = p.sec_as ? F(L.qkvc) : nullptr;
    fd.vr = need_vr ? F(L.vr) : nullptr;   // V^r carried: CL check, CL^r for dW^O
    fd.cl = ws + L.cl;
    fd.check_as = p.sec_as;
    fd.check_cl = p.sec_cl;
    fd.recompute = p.root;
    fd.e_rel = p.e_rel;
    fd.tn_s = stored_threshold(cfg->t_near_inf > 0.f ? cfg->t_near_inf : 1e10f, ABFT_FP32);
    fd.tn_cl = p.tn;
    fd.tc = p.tc;
    fd.faults = faults; fd.n_faults = n_faults; fd.report = report;
    fd.stats = F(L.stats);
    fd.clr = F(L.clr);
    if (es == 2) fd.clri = reinterpret_cast<uint16_t*>(ws + L.clri);
    if (p.sec_o) {  // CL^c of the checked CL for the output projection
      fd.clc = F(L.clc);
      if (es == 2) fd.clci = reinterpret_cast<uint16_t*>(ws + L.clci);
    }
    CK(launch_fused_fwd(fd, s));
  }
  // AS = Q K^T per head (unscaled, before the mask), two-sided checksums
  if (!fused && (stages & ABFT_STAGE_SCORE)) {
    GemmDesc g = base_desc(p, faults, n_faults, report);
    g.M = int(S); g.N = int(S); g.K = int(hd);
    g.nb0 = int(B); g.nb1 = int(nh);
    g.A = ws + L.qkv; g.lda = 3 * H; g.sA0 = S * 3 * H; g.sA1 = hd;
    g.B = ws + L.qkv + H * es; g.ldb = 3 * H; g.sB0 = S * 3 * H; g.sB1 = hd;
    g.C = ws + L.as; g.ldc = S; g.sC0 = nh * S * S; g.sC1 = S * S;
    if (p.sec_as) {
      g.Ac = F(L.qkvc); g.ldac = 3 * H; g.sAc0 = nq * 2 * 3 * H; g.sAc1 = hd; g.Rm = int(R);
      g.Br = F(L.qkvc) + H; g.ldbr = 3 * H; g.sBr0 = nq * 2 * 3 * H; g.sBr1 = hd; g.Rn = int(R);
      g.verify = 2;
    }
    g.causal = cfg->causal ? 1 : 0;
    g.map.op_base = ABFT_OP_AS; g.map.nb1 = int(nh);
    CK(launch_gemm(g, dt, false, Layout::KMajor, Layout::KMajor, Tile::T128x128S1, s));
  }
  // AP = softmax(scale * AS) with column (and row) checksums
  if (!fused && (stages & ABFT_STAGE_SOFTMAX)) {
    SoftmaxDesc sd;
    sd.B = int(B); sd.nh = int(nh); sd.S = int(S); sd.R = int(R); sd.causal = cfg->causal;
    sd.kv_align = 128;
    sd.scale = p.scale;
    sd.AS = ws + L.as; sd.AP = ws + L.ap;
    sd.col_chk = need_apc ? F(L.apc) : nullptr;
    sd.row_chk = p.sec_bwd ? F(L.apr) : nullptr;
    CK(launch_softmax_fwd(sd, dt, s));
  }
  // CL = AP V per head, CL^c = AP^c V, CL^r = AP V^r
  if (!fused && (stages & ABFT_STAGE_CONTEXT)) {
    GemmDesc g = base_desc(p, faults, n_faults, report);
    g.M = int(S); g.N = int(hd); g.K = int(S);
    g.nb0 = int(B); g.nb1 = int(nh);
    g.A = ws + L.ap; g.lda = S; g.sA0 = nh * S * S; g.sA1 = S * S;
    g.B = ws + L.qkv + 2 * H * es; g.ldb = 3 * H; g.sB0 = S * 3 * H; g.sB1 = hd;
    g.C = ws + L.cl; g.ldc = H; g.sC0 = S * H; g.sC1 = hd;
    if (need_apc) {
      g.Ac = F(L.apc); g.ldac = S; g.sAc0 = nh * nq * 2 * S; g.sAc1 = nq * 2 * S; g.Rm = int(R);
      g.Cc = F(L.clc); g.ldcc = H; g.sCc0 = nq * 2 * H; g.sCc1 = hd;
    }
    if (need_vr) {
      g.Br = F(L.vr); g.ldbr = 2 * nh; g.sBr0 = S * 2 * nh; g.sBr1 = 2; g.Rn = int(hd);
      g.Cr = F(L.clr); g.ldcr = 2 * nh; g.sCr0 = S * 2 * nh; g.sCr1 = 2;
    }
    if (p.sec_cl) g.verify = 2;
    g.causal = cfg->causal ? 2 : 0;
    g.map.op_base = ABFT_OP_CL; g.map.nb1 = int(nh);
    CK(launch_gemm(g, dt, false, Layout::KMajor, Layout::MNMajor,
                   hd == 64 ? Tile::T128x64 : Tile::T128x128, s));
  }
  // O = CL Wo, O^c = CL^c Wo
  if (stages & ABFT_STAGE_OUT) {
    GemmDesc g = base_desc(p, faults, n_faults, report);
    g.M = int(T); g.N = int(H); g.K = int(H);
    g.A = ws + L.cl; g.lda = H;
    g.B = Wo; g.ldb = H;
    g.C = O; g.ldc = H;
    if (p.sec_o) {
      g.Ac = F(L.clc); g.ldac = H; g.Rm = int(R);
      if (fused && es == 2) {  // the image the fused forward wrote with CL^c
        g.Aci = reinterpret_cast<const uint16_t*>(ws + L.clci); g.ldaci = H;
      }
      g.verify = 1;
    }
    g.map.op_base = ABFT_OP_O; g.map.rows_per_b = int(S);
    CK(launch_gemm(g, dt, false, Layout::KMajor, Layout::MNMajor, proj_tile(), s));
  }
  return ABFT_OK;
}

}  // namespace
}  // namespace abft

extern "C" {

int attn_abft_forward_stages(const attn_abft_config* cfg, const void* X, const void* Wqkv,
                             const void* Wo, void* O, void* workspace, size_t workspace_bytes,
                             const abft_fault* faults, int32_t n_faults, abft_report* report,
                             uint32_t stages, void* stream) {
  Dims d;
  int st = validate(cfg, &d);
  if (st != ABFT_OK) return st;
  if (!X || !Wqkv || !Wo || !O || !workspace || !report || n_faults < 0 ||
      (n_faults > 0 && !faults))
    return ABFT_ERR_INVALID;
  const Layout_ L = layout_for(cfg, d);
  if (workspace_bytes < L.total) return ABFT_ERR_WORKSPACE;
  if ((st = check_device()) != ABFT_OK) return st;
  return forward_impl(cfg, d, L, make_params(cfg, d), X, Wqkv, Wo, O,
                      static_cast<char*>(workspace), faults, n_faults, report, stages,
                      static_cast<hipStream_t>(stream));
}

int attn_abft_backward_stages(const attn_abft_config* cfg, const void* dO, const void* X,
                              const void* Wqkv, const void* Wo, void* workspace,
                              size_t workspace_bytes, void* dX, float* dWqkv, float* dWo,
                              const abft_fault* faults, int32_t n_faults, abft_report* report,
                              uint32_t stages, void* stream) {
  Dims d;
  int st = validate(cfg, &d);
  if (st != ABFT_OK) return st;
  if (!dO || !X || !Wqkv || !Wo || !workspace || !dX || !dWqkv || !dWo || !report ||
      n_faults < 0 || (n_faults > 0 && !faults))
    return ABFT_ERR_INVALID;
  const Layout_ L = layout_for(cfg, d);
  if (workspace_bytes < L.total) return ABFT_ERR_WORKSPACE;
  if ((st = check_device()) != ABFT_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Params p = make_params(cfg, d);
  const int dt = cfg->dtype;
  char* ws = static_cast<char*>(workspace);
  auto F = [&](size_t off) { return reinterpret_cast<float*>(ws + off); };
  const int64_t B = d.B, S = d.S, H = d.H, nh = d.nh, hd = d.d, R = d.R, nq = d.nq, T = d.T;
  const size_t es = d.es;
  const bool pb = p.sec_bwd;

  const bool fused = (cfg->flags & ABFT_FLAG_FUSED) != 0;
  // dO^c (Sec. 4.6), with the report cleared in the same launch
  {
    EncodeJob e[1];
    int nj = 0;
    if ((stages & ABFT_STAGE_ENCODE) && pb) {
      EncodeJob& j = e[nj++];
      j.A = dO; j.batch = B; j.rows = S; j.cols = H; j.ld = H; j.batch_stride = S * H;
      j.Rb = int(R); j.Cb = int(hd); j.col_chk = F(L.doc);
      if (es == 2) { j.col_img = reinterpret_cast<uint16_t*>(ws + L.doci); j.ldci = H; }
    }
    CK(launch_encode_jobs(e, nj, dt, (cfg->flags & ABFT_FLAG_REPORT_APPEND) ? nullptr : report,
                          s));
  }

  // dCL = dO Wo^T, dCL^c = dO^c Wo^T, and dWo = CL^T dO (independent: one
  // launch when both qualify)
  GemmDesc gdcl, gdwo;
  if (stages & ABFT_STAGE_DCL) {
    GemmDesc& g = gdcl;
    g = base_desc(p, faults, n_faults, report);
    g.M = int(T); g.N = int(H); g.K = int(H);
    g.A = dO; g.lda = H;
    g.B = Wo; g.ldb = H;
    g.C = ws + L.dcl; g.ldc = H;
    if (pb) {
      g.Ac = F(L.doc); g.ldac = H; g.Rm = int(R);
      if (es == 2) { g.Aci = reinterpret_cast<const uint16_t*>(ws + L.doci); g.ldaci = H; }
      g.Cc = F(L.dclc); g.ldcc = H;
      g.verify = 1;
    }
    g.map.op_base = ABFT_OP_DCL; g.map.rows_per_b = int(S); g.map.head_cols = int(hd);
  }
  // dWo = CL^T dO, column checksums over head blocks of rows from CL^r
  if (stages & ABFT_STAGE_DWO) {
    GemmDesc& g = gdwo;
    g = base_desc(p, faults, n_faults, report);
    g.M = int(H); g.N = int(H); g.K = int(T);
    g.A = ws + L.cl; g.lda = H;
    g.B = dO; g.ldb = H;
    g.C = dWo; g.ldc = H;
    if (pb) {
      g.Ac = F(L.clr); g.ldac = 2 * nh; g.Rm = int(hd);
      if (fused && es == 2) {  // the image the fused forward wrote with CL^r
        g.Aci = reinterpret_cast<const uint16_t*>(ws + L.clri); g.ldaci = T;
      }
      g.verify = 1;
    }
    g.map.op_base = ABFT_OP_DWO;
  }
  CK(wgrad_with_proj((stages & ABFT_STAGE_DWO) ? &gdwo : nullptr,
                     (stages & ABFT_STAGE_DCL) ? &gdcl : nullptr, dt, F(L.skp), F(L.skc), s));
  // after a fused forward (no scores kept): the fused backward core, from
  // the forward's softmax statistics, in two launches: the query pass (dQ,
  // and D per query) and the key pass (dK and dV); each forms the row
  // checksums over the head dims that it needs (K^r; Q^r and dCL^r) from
  // the tiles it stages; nothing score-shaped is stored (dQ^c, dK^c and
  // dV^c are encoded at the dX stage)
  if (fused) {
    const uint32_t st_q = ABFT_STAGE_CORE_BWD | ABFT_STAGE_SOFTMAX_BWD | ABFT_STAGE_DQ;
    const uint32_t st_kv = ABFT_STAGE_CORE_BWD | ABFT_STAGE_DV | ABFT_STAGE_DK;
    FusedBwdDesc fd;
    fd.B = int(B); fd.nh = int(nh); fd.S = int(S); fd.H = int(H); fd.D = int(hd); fd.R = int(R);
    fd.causal = cfg->causal;
    fd.scale = p.scale;
    fd.qkv = ws + L.qkv;
    fd.qkvc = pb ? F(L.qkvc) : nullptr;
    fd.dclc = pb ? F(L.dclc) : nullptr;
    fd.cl = ws + L.cl;
    fd.dcl = ws + L.dcl;
    fd.stats = F(L.stats);
    fd.drow = F(L.drow);
    fd.dqkv = ws + L.dqkv; fd.ld = 3 * H;
    fd.check = pb ? 1 : 0;
    fd.recompute = p.root ? 1 : 0;
    fd.e_rel = p.e_rel;
    fd.tn_s = stored_threshold(cfg->t_near_inf > 0.f ? cfg->t_near_inf : 1e10f, ABFT_FP32);
    fd.tn = p.tn;
    fd.tc = p.tc;
    fd.faults = faults; fd.n_faults = n_faults; fd.report = report;
    if (stages & st_q) CK(launch_fused_bwd_q(fd, s));
    if (stages & st_kv) CK(launch_fused_bwd_kv(fd, s));
  }
  // dAP = dCL_h V_h^T, dAP^c = dCL_h^c V_h^T
  if (!fused && (stages & ABFT_STAGE_DAP)) {
    GemmDesc g = base_desc(p, faults, n_faults, report);
    g.M = int(S); g.N = int(S); g.K = int(hd);
    g.nb0 = int(B); g.nb1 = int(nh);
    g.A = ws + L.dcl; g.lda = H; g.sA0 = S * H; g.sA1 = hd;
    g.B = ws + L.qkv + 2 * H * es; g.ldb = 3 * H; g.sB0 = S * 3 * H; g.sB1 = hd;
    g.C = ws + L.as; g.ldc = S; g.sC0 = nh * S * S; g.sC1 = S * S;
    if (pb) {
      g.Ac = F(L.dclc); g.ldac = H; g.sAc0 = nq * 2 * H; g.sAc1 = hd; g.Rm = int(R);
      g.verify = 1;
    }
    g.causal = cfg->causal ? 1 : 0;
    g.map.op_base = ABFT_OP_DAP; g.map.nb1 = int(nh);
    CK(launch_gemm(g, dt, false, Layout::KMajor, Layout::KMajor, Tile::T128x128S1, s));
  }
  const Tile td = hd == 64 ? Tile::T128x64 : Tile::T128x128;
  // dV = AP^T dCL_h, column checksums over key blocks from AP^r
  if (!fused && (stages & ABFT_STAGE_DV)) {
    GemmDesc g = base_desc(p, faults, n_faults, report);
    g.M = int(S); g.N = int(hd); g.K = int(S);
    g.nb0 = int(B); g.nb1 = int(nh);
    g.A = ws + L.ap; g.lda = S; g.sA0 = nh * S * S; g.sA1 = S * S;
    g.B = ws + L.dcl; g.ldb = H; g.sB0 = S * H; g.sB1 = hd;
    g.C = ws + L.dqkv + 2 * H * es; g.ldc = 3 * H; g.sC0 = S * 3 * H; g.sC1 = hd;
    if (pb) {
      g.Ac = F(L.apr); g.ldac = nq * 2; g.sAc0 = nh * S * nq * 2; g.sAc1 = S * nq * 2;
      g.Rm = int(R);
      g.Cc = F(L.dqkvc) + 2 * H; g.ldcc = 3 * H; g.sCc0 = nq * 2 * 3 * H; g.sCc1 = hd;
      g.verify = 1;
    }
    g.causal = cfg->causal ? 3 : 0;
    g.map.op_base = ABFT_OP_DV; g.map.nb1 = int(nh);
    CK(launch_gemm(g, dt, false, Layout::MNMajor, Layout::MNMajor, td, s));
  }
  // dAS = scale * AP * (dAP - rowdot), with column and row checksums
  if (!fused && (stages & ABFT_STAGE_SOFTMAX_BWD)) {
    SoftmaxDesc sd;
    sd.B = int(B); sd.nh = int(nh); sd.S = int(S); sd.R = int(R); sd.causal = cfg->causal;
    sd.kv_align = 128;
    sd.scale = p.scale;
    sd.AP = ws + L.ap; sd.dAP = ws + L.as; sd.dAS = ws + L.das;
    sd.col_chk = pb ? F(L.dasc) : nullptr;
    sd.row_chk = pb ? F(L.dasr) : nullptr;
    CK(launch_softmax_bwd(sd, dt, s));
  }
  // dQ = dAS K_h, dQ^c = dAS^c K_h
  if (!fused && (stages & ABFT_STAGE_DQ)) {
    GemmDesc g = base_desc(p, faults, n_faults, report);
    g.M = int(S); g.N = int(hd); g.K = int(S);
    g.nb0 = int(B); g.nb1 = int(nh);
    g.A = ws + L.das; g.lda = S; g.sA0 = nh * S * S; g.sA1 = S * S;
    g.B = ws + L.qkv + H * es; g.ldb = 3 * H; g.sB0 = S * 3 * H; g.sB1 = hd;
    g.C = ws + L.dqkv; g.ldc = 3 * H; g.sC0 = S * 3 * H; g.sC1 = hd;
    if (pb) {
      g.Ac = F(L.dasc); g.ldac = S; g.sAc0 = nh * nq * 2 * S; g.sAc1 = nq * 2 * S; g.Rm = int(R);
      g.Cc = F(L.dqkvc); g.ldcc = 3 * H; g.sCc0 = nq * 2 * 3 * H; g.sCc1 = hd;
      g.verify = 1;
    }
    g.causal = cfg->causal ? 2 : 0;
    g.map.op_base = ABFT_OP_DQ; g.map.nb1 = int(nh);
    CK(launch_gemm(g, dt, false, Layout::KMajor, Layout::MNMajor, td, s));
  }
  // dK = dAS^T Q_h, column checksums over key blocks from dAS^r
  if (!fused && (stages & ABFT_STAGE_DK)) {
    GemmDesc g = base_desc(p, faults, n_faults, report);
    g.M = int(S); g.N = int(hd); g.K = int(S);
    g.nb0 = int(B); g.nb1 = int(nh);
    g.A = ws + L.das; g.lda = S; g.sA0 = nh * S * S; g.sA1 = S * S;
    g.B = ws + L.qkv; g.ldb = 3 * H; g.sB0 = S * 3 * H; g.sB1 = hd;
    g.C = ws + L.dqkv + H * es; g.ldc = 3 * H; g.sC0 = S * 3 * H; g.sC1 = hd;
    if (pb) {
      g.Ac = F(L.dasr); g.ldac = nq * 2; g.sAc0 = nh * S * nq * 2; g.sAc1 = S * nq * 2;
      g.Rm = int(R);
      g.Cc = F(L.dqkvc) + H; g.ldcc = 3 * H; g.sCc0 = nq * 2 * 3 * H; g.sCc1 = hd;
      g.verify = 1;
    }
    g.causal = cfg->causal ? 3 : 0;
    g.map.op_base = ABFT_OP_DK; g.map.nb1 = int(nh);
    CK(launch_gemm(g, dt, false, Layout::MNMajor, Layout::MNMajor, td, s));
  }
  // dX = dQKV Wqkv^T, dX^c = dQKV^c Wqkv^T, and dWqkv = X^T dQKV (independent:
  // one launch when both qualify)
  if ((stages & ABFT_STAGE_DX) && fused && pb) {
    // the fused core writes no checksums: dQKV^c from the checked dQKV
    EncodeJob e;
    e.A = ws + L.dqkv; e.batch = B; e.rows = S; e.cols = 3 * H; e.ld = 3 * H;
    e.batch_stride = S * 3 * H; e.Rb = int(R); e.Cb = int(hd);
    e.col_chk = F(L.dqkvc); e.ldcc = 3 * H;
    if (es == 2) { e.col_img = reinterpret_cast<uint16_t*>(ws + L.dqkvci); e.ldci = 3 * H; }
    CK(launch_encode_jobs(&e, 1, dt, nullptr, s));
  }
  // dWqkv: column checksums over head blocks of rows from X^r
  GemmDesc gdwq, gdx;
  if (stages & ABFT_STAGE_DWQKV) {
    GemmDesc& g = gdwq;
    g = base_desc(p, faults, n_faults, report);
    g.M = int(H); g.N = int(3 * H); g.K = int(T);
    g.A = X; g.lda = H;
    g.B = ws + L.dqkv; g.ldb = 3 * H;
    g.C = dWqkv; g.ldc = 3 * H;
    if (pb) {
      g.Ac = F(L.xr); g.ldac = 2 * nh; g.Rm = int(hd);
      if (es == 2) { g.Aci = reinterpret_cast<const uint16_t*>(ws + L.xri); g.ldaci = T; }
      g.verify = 1;
    }
    g.map.op_base = ABFT_OP_DWQ; g.map.op_span = int(H);
  }
  if (stages & ABFT_STAGE_DX) {
    GemmDesc& g = gdx;
    g = base_desc(p, faults, n_faults, report);
    g.M = int(T); g.N = int(H); g.K = int(3 * H);
    g.A = ws + L.dqkv; g.lda = 3 * H;
    g.B = Wqkv; g.ldb = 3 * H;
    g.C = dX; g.ldc = H;
    if (pb) {
      g.Ac = F(L.dqkvc); g.ldac = 3 * H; g.Rm = int(R);
      if (fused && es == 2) {  // the image the encode above wrote
        g.Aci = reinterpret_cast<const uint16_t*>(ws + L.dqkvci); g.ldaci = 3 * H;
      }
      g.verify = 1;
    }
    g.map.op_base = ABFT_OP_DX; g.map.rows_per_b = int(S);
  }
  CK(wgrad_with_proj((stages & ABFT_STAGE_DWQKV) ? &gdwq : nullptr,
                     (stages & ABFT_STAGE_DX) ? &gdx : nullptr, dt, F(L.skp), F(L.skc), s));
  return ABFT_OK;
}

int attn_abft_forward(const attn_abft_config* cfg, const void* X, const void* Wqkv,
                      const void* Wo, void* O, void* workspace, size_t workspace_bytes,
                      const abft_fault* faults, int32_t n_faults, abft_report* report,
                      void* stream) {
  return attn_abft_forward_stages(cfg, X, Wqkv, Wo, O, workspace, workspace_bytes, faults,
                                  n_faults, report, ABFT_STAGE_ALL, stream);
}

int attn_abft_backward(const attn_abft_config* cfg, const void* dO, const void* X,
                       const void* Wqkv, const void* Wo, void* workspace,
                       size_t workspace_bytes, void* dX, float* dWqkv, float* dWo,
                       const abft_fault* faults, int32_t n_faults, abft_report* report,
                       void* stream) {
  return attn_abft_backward_stages(cfg, dO, X, Wqkv, Wo, workspace, workspace_bytes, dX, dWqkv,
                                   dWo, faults, n_faults, report, ABFT_STAGE_ALL, stream);
}

int encode_checksums(const void* A, int32_t dtype, int64_t batch, int64_t rows, int64_t cols,
                     int64_t ld, int64_t batch_stride, int32_t block_rows, int32_t block_cols,
                     float* col_chk, float* row_chk, void* stream) {
  if (!A || batch < 0 || rows < 0 || cols < 0 || ld < cols) return ABFT_ERR_INVALID;
  if (dtype != ABFT_BF16 && dtype != ABFT_FP32) return ABFT_ERR_UNSUPPORTED;
  if (col_chk && (block_rows < 1 || rows % block_rows)) return ABFT_ERR_INVALID;
  if (row_chk && (block_cols < 1 || cols % block_cols)) return ABFT_ERR_INVALID;
  if (!col_chk && !row_chk) return ABFT_OK;
  int st = check_device();
  if (st != ABFT_OK) return st;
  int Rb = block_rows;
  if (!col_chk) {  // only row checksums: any row block works; pick one with many workgroups
    Rb = 1;
    while (Rb < 32 && rows % (2 * Rb) == 0) Rb *= 2;
  }
  CK(launch_encode(A, dtype, batch, rows, cols, ld, batch_stride, Rb, block_cols, col_chk, row_chk,
                   static_cast<hipStream_t>(stream)));
  return ABFT_OK;
}

int verify_and_correct(void* C, int32_t dtype, int64_t batch, int64_t rows, int64_t cols,
                       int64_t ld, int64_t batch_stride, int32_t block_rows, int32_t block_cols,
                       float* col_chk, float* row_chk, float t_near_inf, float t_correct,
                       float e_rel, int32_t op_tag, abft_report* report, void* stream) {
  if (!C || !col_chk || !report || batch < 0 || rows < 0 || cols < 0 || ld < cols)
    return ABFT_ERR_INVALID;
  if (dtype != ABFT_BF16 && dtype != ABFT_FP32) return ABFT_ERR_UNSUPPORTED;
  if (block_rows < 1 || rows % block_rows) return ABFT_ERR_INVALID;
  if (row_chk && (block_cols < 1 || cols % block_cols)) return ABFT_ERR_INVALID;
  if (!(t_near_inf >= 0.f) || !(t_correct >= 0.f) || !(e_rel >= 0.f)) return ABFT_ERR_INVALID;
  if (size_t(block_rows) * (row_chk ? cols / block_cols : 0) + (row_chk ? cols : 0) >
      size_t(150 * 1024 / 4))
    return ABFT_ERR_UNSUPPORTED;
  int st = check_device();
  if (st != ABFT_OK) return st;
  const float er = e_rel > 0.f ? e_rel : (dtype == ABFT_FP32 ? std::ldexp(1.f, -13)
                                                              : std::ldexp(1.f, -4));
  const float tn = stored_threshold(t_near_inf > 0.f ? t_near_inf : 1e10f, dtype);
  const float tc = t_correct > 0.f ? t_correct : 1e5f;
  CK(launch_verify(C, dtype, batch, rows, cols, ld, batch_stride, block_rows, block_cols, col_chk,
                   row_chk, tn, tc, er, op_tag, report, static_cast<hipStream_t>(stream)));
  return ABFT_OK;
}

const char* attn_abft_strerror(int status) {
  switch (status) {
    case ABFT_OK: return "ok";
    case ABFT_ERR_INVALID: return "invalid argument";
    case ABFT_ERR_UNSUPPORTED: return "unsupported configuration or device";
    case ABFT_ERR_HIP: return "HIP launch error";
    case ABFT_ERR_WORKSPACE: return "workspace too small";
  }
  return "unknown status";
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Allocation-free forward: the fused protected forward with its workspace in
// a buffer of the library's own, for callers that cannot allocate device
// memory (code under graph capture, tight serving loops).
namespace abft {

constexpr size_t NOALLOC_SCRATCH_BYTES = size_t(64) << 20;

// The buffer: one copy on every device the library runs on, held until the
// process ends. In host code `scratch` names a host-side stand-in; kernels
// get the device address that hipGetSymbolAddress returns for the current
// device.
static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

namespace {

// Device address of `scratch` on the current device, looked up once per
// device with that device current; nullptr if the lookup fails.
char* scratch_on_current_device() {
  static std::mutex mu;
  static char* addr[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lk(mu);
  if (addr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr)
      return nullptr;
    addr[dev] = static_cast<char*>(ptr);
  }
  return addr[dev];
}

}  // namespace
}  // namespace abft

extern "C" {

int attn_abft_forward_noalloc(const attn_abft_config* cfg, const void* X, const void* Wqkv,
                              const void* Wo, void* O, const abft_fault* faults,
                              int32_t n_faults, abft_report* report, void* stream) {
  Dims d;
  int st = validate(cfg, &d);
  if (st != ABFT_OK) return st;
  if (!(cfg->flags & ABFT_FLAG_FUSED)) return ABFT_ERR_UNSUPPORTED;
  if (!X || !Wqkv || !Wo || !O || !report || n_faults < 0 || (n_faults > 0 && !faults))
    return ABFT_ERR_INVALID;
  const Layout_ L = make_layout_fused_forward(d);
  if (L.total > NOALLOC_SCRATCH_BYTES) return ABFT_ERR_WORKSPACE;
  if ((st = check_device()) != ABFT_OK) return st;
  char* ws = scratch_on_current_device();
  if (ws == nullptr) return ABFT_ERR_HIP;
  Params p = make_params(cfg, d);
  p.sec_bwd = false;  // nothing is kept for a backward
  return forward_impl(cfg, d, L, p, X, Wqkv, Wo, O, ws, faults, n_faults, report,
                      ABFT_STAGE_ALL, static_cast<hipStream_t>(stream));
}

}  // extern "C"
