// Host side of libks: argument validation, the tiling planner and plan cache,
// the C ABI entry points and the chain driver.
//
// Every check runs on the host before anything is enqueued, so each error path
// can be exercised without a GPU.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <unordered_map>

#include "../../include/ks.h"
#include "ks_chain_fused.h"
#include "ks_direct_index.h"
#include "ks_internal.h"

namespace ks {
namespace {

thread_local int g_last_hip_error = 0;
thread_local int g_forced_variant = -1;
thread_local int g_chain_fusion = -1;  // -1 automatic, 0 never fuse a chain

constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;

// Bytes per element of X and K_values (in) and of Y and bias (out): FP8
// inputs (E4M3) produce bfloat16 outputs.
int elem_size(int dtype) { return dtype == F32 ? 4 : 2; }
int in_size(int dtype) { return dtype == FP8 ? 1 : elem_size(dtype); }
int out_size(int dtype) { return dtype == FP8 ? 2 : elem_size(dtype); }

bool mul_ok(int64_t x, int64_t y, int64_t* out) { return !__builtin_mul_overflow(x, y, out); }

// Pattern sizes with overflow checks.
struct Dims {
  int64_t N = 0, M = 0, nnz = 0;
};

ks_status_t check_pattern(int64_t a, int64_t b, int64_t c, int64_t d, Dims* dims) {
  if (a < 1 || b < 1 || c < 1 || d < 1) return KS_ERR_INVALID_PATTERN;
  int64_t ad, N, M, nnz;
  if (!mul_ok(a, d, &ad) || !mul_ok(ad, c, &N) || !mul_ok(ad, b, &M) || !mul_ok(M, c, &nnz))
    return KS_ERR_INVALID_PATTERN;
  dims->N = N;
  dims->M = M;
  dims->nnz = nnz;
  return KS_OK;
}

bool overlaps(const void* p, int64_t pbytes, const void* q, int64_t qbytes) {
  if (pbytes <= 0 || qbytes <= 0) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(p), a1 = a0 + (uintptr_t)pbytes;
  const uintptr_t b0 = reinterpret_cast<uintptr_t>(q), b1 = b0 + (uintptr_t)qbytes;
  return a0 < b1 && b0 < a1;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ---------------------------------------------------------------------------
// Planner.  Each variant planner fills `pl` and returns true when the variant
// can run the problem.
// ---------------------------------------------------------------------------

bool plan_generic(const Problem& p, Plan* pl) {
  pl->variant = V_GENERIC;
  const int64_t total = (int64_t)p.batch * p.M;
  const int64_t blocks = (total + 255) / 256;
  pl->block = 256;
  pl->grid = (unsigned)std::max<int64_t>(1, std::min<int64_t>(blocks, 256 * 64));
  return true;
}

// Batch-size-last VALU streaming: b, c <= 16; 16-byte vectors along the batch
// when the batch is a multiple of the vector width and the buffers are
// 16-byte aligned, single elements otherwise.
bool plan_valu_bsl(const Problem& p, bool al16, Plan* pl) {
  if (p.layout != BSL || p.b > kValuMaxBC || p.c > kValuMaxBC) return false;
  if ((int64_t)p.a * p.d > 65535) return false;
  const int vec16 = 16 / elem_size(p.dtype);
  const int vec = (al16 && p.batch % vec16 == 0) ? vec16 : 1;
  const int u = valu_bsl_unroll(p.b, p.c);
  const int nvec = p.batch / vec;
  pl->variant = V_VALU_BSL;
  pl->vec = vec;
  pl->unroll = u;
  pl->block = 256;
  pl->grid = (unsigned)((nvec + 256 * u - 1) / (256 * u));
  return true;
}

// Batch-size-first VALU: b, c <= 16; a thread owns V consecutive j, V the
// largest power of two dividing d that fits a 16-byte vector (given alignment).
bool plan_valu_bsf(const Problem& p, bool al16, Plan* pl) {
  if (p.layout != BSF || p.b > kValuMaxBC || p.c > kValuMaxBC) return false;
  const int vec16 = 16 / elem_size(p.dtype);
  int v = 1;
  if (al16)
    while (v * 2 <= vec16 && p.d % (v * 2) == 0) v *= 2;
  const int64_t total = (int64_t)p.batch * p.a * (p.d / v);
  const int64_t blocks = (total + 255) / 256;
  if (blocks > 0x7fffffff) return false;
  pl->variant = V_VALU_BSF;
  pl->vec = v;
  pl->block = 256;
  pl->grid = (unsigned)blocks;
  return true;
}

}  // namespace
bool plan_direct(const Problem& p, bool al16, Plan* pl);
bool plan_staged(const Problem& p, bool al16, Plan* pl);
bool plan_dma(const Problem& p, bool al16, Plan* pl);
bool plan_masked(const Problem& p, Plan* pl);
bool plan_fp8(const Problem& p, Plan* pl);
namespace {

bool plan_variant(int v, const Problem& p, bool al16, Plan* pl) {
  switch (v) {
    case V_GENERIC: return plan_generic(p, pl);
    case V_VALU_BSL: return plan_valu_bsl(p, al16, pl);
    case V_VALU_BSF: return plan_valu_bsf(p, al16, pl);
    case V_DIRECT: return plan_direct(p, al16, pl);
    case V_STAGED: return plan_staged(p, al16, pl);
    case V_DMA: return plan_dma(p, al16, pl);
    case V_MASKED: return plan_masked(p, pl);
    case V_FP8: return plan_fp8(p, pl);
    default: return false;
  }
}

// Automatic choice: MFMA block GEMM when b and c make each (i, j) block a real
// dense contraction (batch-size-first through LDS: DMA-fed for d <= 16,
// register-staged beyond; register-direct for batch-size-last and small
// batch-size-first problems); VALU kernels for small blocks; the masked
// register-direct kernel for larger blocks the others cannot take (b or c not
// a multiple of 16, odd batches, unaligned buffers); the generic kernel only
// when forced.
bool plan_auto(const Problem& p, bool al16, Plan* pl) {
  if (p.dtype == FP8) return plan_fp8(p, pl);  // the only FP8 kernel
  // Batch-size-first with d <= 2: the DMA kernel from 8 MB of X + Y up
  // (measured: below that the register-direct items' shorter latency wins).
  const int64_t xy_bytes = (int64_t)p.batch * (p.N + p.M) * (p.dtype == F32 ? 4 : 2);
  if (p.layout == BSF && (p.d >= 4 || xy_bytes >= (8 << 20)) && plan_dma(p, al16, pl)) return true;
  if (p.layout == BSF && p.d >= 4 && plan_staged(p, al16, pl)) return true;
  // Batch-size-last: the DMA kernel for fp32, and for 16-bit types with b a
  // power of two from 32 and c of 32 or 64 (measured on the sampled sweep
  // points: fp32 sweep median 0.437 -> 0.549 at batch 25088 and 0.367 ->
  // 0.412 at 4096; for 16-bit types elsewhere, where the k-groups of b = 48
  // or 96 re-read X or the stages of 32 values of l leave too few tiles, the
  // register-direct kernel is faster).
  const bool bsl_dma = p.dtype == F32 || ((p.b & (p.b - 1)) == 0 && p.b >= 32 && p.c <= 64);
  if (p.layout == BSL && bsl_dma && plan_dma(p, al16, pl)) return true;
  if (plan_direct(p, al16, pl)) return true;
  if (p.layout == BSL && plan_valu_bsl(p, al16, pl)) return true;
  if (p.layout == BSF && plan_valu_bsf(p, al16, pl)) return true;
  if (plan_masked(p, pl)) return true;
  return plan_generic(p, pl);
}

struct PlanKey {
  int64_t a, b, c, d, batch;
  int layout, dtype, al16, align, forced;
  bool operator==(const PlanKey& o) const {
    return a == o.a && b == o.b && c == o.c && d == o.d && batch == o.batch && layout == o.layout &&
           dtype == o.dtype && al16 == o.al16 && align == o.align && forced == o.forced;
  }
};
struct PlanKeyHash {
  size_t operator()(const PlanKey& k) const {
    uint64_t h = 1469598103934665603ull;
    const int64_t v[10] = {k.a, k.b, k.c, k.d, k.batch, k.layout, k.dtype, k.al16, k.align, k.forced};
    for (int64_t x : v) { h ^= (uint64_t)x; h *= 1099511628211ull; }
    return (size_t)h;
  }
};

std::mutex g_plan_mu;
std::unordered_map<PlanKey, Plan, PlanKeyHash>* g_plans = nullptr;

// Returns false when a forced variant cannot run the problem.
bool get_plan(const Problem& p, bool al16, Plan* out) {
  const int forced = g_forced_variant;
  PlanKey key{p.a, p.b, p.c, p.d, p.batch, p.layout, p.dtype, al16 ? 1 : 0, p.align, forced};
  {
    std::lock_guard<std::mutex> lk(g_plan_mu);
    if (!g_plans) g_plans = new std::unordered_map<PlanKey, Plan, PlanKeyHash>();
    auto it = g_plans->find(key);
    if (it != g_plans->end()) { *out = it->second; return true; }
  }
  Plan pl;
  bool ok = forced >= 0 ? ((p.dtype == FP8) == (forced == V_FP8) && plan_variant(forced, p, al16, &pl))
                        : plan_auto(p, al16, &pl);
  if (!ok) return false;
  std::lock_guard<std::mutex> lk(g_plan_mu);
  (*g_plans)[key] = pl;
  *out = pl;
  return true;
}

hipError_t launch(const Problem& p, const Plan& pl, hipStream_t s) {
  switch (pl.variant) {
    case V_GENERIC: return launch_generic(p, pl, s);
    case V_VALU_BSL: return launch_valu_bsl(p, pl, s);
    case V_VALU_BSF: return launch_valu_bsf(p, pl, s);
    case V_DIRECT: return launch_direct(p, pl, s);
    case V_STAGED: return launch_staged(p, pl, s);
    case V_DMA: return launch_dma(p, pl, s);
    case V_MASKED: return launch_masked(p, pl, s);
    case V_FP8: return launch_fp8(p, pl, s);
    default: return hipErrorInvalidValue;
  }
}

// Full validation of a single-factor call; fills `p` on success.
ks_status_t validate(int64_t a, int64_t b, int64_t c, int64_t d, const void* kv, const void* x, void* y,
                     int64_t batch, int layout, int dtype, Problem* p, bool* empty) {
  Dims dm;
  ks_status_t st = check_pattern(a, b, c, d, &dm);
  if (st != KS_OK) return st;
  if (layout != KS_LAYOUT_BSF && layout != KS_LAYOUT_BSL) return KS_ERR_UNSUPPORTED;
  if (dtype != KS_F32 && dtype != KS_BF16 && dtype != KS_F16 && dtype != KS_FP8_E4M3) return KS_ERR_UNSUPPORTED;
  if (batch < 0) return KS_ERR_INVALID_ARG;
  if (kv == nullptr) return KS_ERR_INVALID_ARG;
  *empty = (batch == 0);
  if (*empty) return KS_OK;
  if (x == nullptr || y == nullptr) return KS_ERR_INVALID_ARG;
  int64_t xe, ye;
  if (!mul_ok(batch, dm.N, &xe) || !mul_ok(batch, dm.M, &ye)) return KS_ERR_UNSUPPORTED;
  if (xe > kMaxElems || ye > kMaxElems || dm.nnz > kMaxElems || batch > kMaxElems) return KS_ERR_UNSUPPORTED;
  const int si = in_size(dtype), so = out_size(dtype);
  if (overlaps(x, xe * si, y, ye * so)) return KS_ERR_ALIAS;
  if (overlaps(kv, dm.nnz * si, y, ye * so)) return KS_ERR_ALIAS;
  p->a = (int)a; p->b = (int)b; p->c = (int)c; p->d = (int)d;
  p->batch = (int)batch;
  p->N = (int)dm.N; p->M = (int)dm.M;
  p->layout = layout; p->dtype = dtype;
  p->kv = kv; p->x = x; p->y = y;
  const uintptr_t bits = reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(y) | 16;
  p->align = (int)(bits & (~bits + 1));  // lowest set bit: 1, 2, 4, 8 or 16
  p->bias = nullptr;
  p->act = 0;
  return KS_OK;
}

bool all_aligned(const Problem& p) { return aligned16(p.kv) && aligned16(p.x) && aligned16(p.y); }

ks_status_t run_one(const Problem& p, hipStream_t s) {
  Plan pl;
  if (!get_plan(p, all_aligned(p), &pl)) return KS_ERR_UNSUPPORTED;
  hipError_t e = launch(p, pl, s);
  if (e != hipSuccess) {
    g_last_hip_error = (int)e;
    return KS_ERR_HIP;
  }
  return KS_OK;
}

// Name of the kernel instance a plan launches, written like the demangled
// symbol without namespace, spaces or parameter list (profiler summaries are
// matched against it).
std::string kernel_name(const Problem& p, const Plan& pl) {
  static const char* tnames[] = {"float", "unsigned short", "_Float16", "unsigned char"};
  const char* t = tnames[p.dtype];
  const int m = p.b > p.c ? p.b : p.c;
  const int mx = m <= 2 ? 2 : (m <= 4 ? 4 : (m <= 8 ? 8 : 16));
  const char* epi = has_epilogue(p) ? "true" : "false";  // direct / masked instances with the epilogue
  char buf[160];
  switch (pl.variant) {
    case V_GENERIC: snprintf(buf, sizeof buf, "ks_generic_kernel<%s>", t); break;
    case V_VALU_BSL:
      snprintf(buf, sizeof buf, "ks_valu_bsl_kernel<%s,%d,%d,%d,%d>", t, pl.vec, mx, mx, valu_bsl_unroll(p.b, p.c));
      break;
    case V_VALU_BSF: snprintf(buf, sizeof buf, "ks_valu_bsf_kernel<%s,%d,%d,%d>", t, pl.vec, mx, mx); break;
    case V_DIRECT: {
      int nch = 0;
      bool tail = false;
      if (direct_c_specialised(p.dtype == F32 ? 4 : 2, p.c, &nch, &tail))
        snprintf(buf, sizeof buf, "ks_direct_c_kernel<%s,%d,%d,%s,%d,%d,%s,%s>", t, p.layout, pl.vec,
                 pl.unroll ? "true" : "false", pl.waves_m, nch, tail ? "true" : "false", epi);
      else
        snprintf(buf, sizeof buf, "ks_direct_kernel<%s,%d,%d,%s,%d,%s>", t, p.layout, pl.vec,
                 pl.unroll ? "true" : "false", pl.waves_m, epi);
      break;
    }
    case V_STAGED:
      snprintf(buf, sizeof buf, "ks_staged_kernel<%s,%d,%d,%s,%d,%d>", t, p.layout, pl.vec,
               pl.unroll ? "true" : "false", pl.waves_m, pl.cps);
      break;
    case V_DMA:
      if (p.layout == BSL) {
        snprintf(buf, sizeof buf, "ks_dma_bsl_kernel<%s,%d,%d,%s>", t, pl.waves_m, pl.rs, epi);
        break;
      }
      // DMA instructions per wavefront per stage: 16*rs rows of lch*d*esize
      // bytes over four wavefronts of 64 16-byte lanes.
      snprintf(buf, sizeof buf, "ks_dma_kernel<%s,%d,%s,%d,%d,%d,%d>", t, pl.vec, pl.unroll ? "true" : "false",
               pl.waves_m, pl.cps, (int)(pl.rs * pl.nt * pl.lch * p.d * (p.dtype == F32 ? 4 : 2) / 256), pl.nt);
      break;
    case V_MASKED: snprintf(buf, sizeof buf, "ks_masked_kernel<%s,%d,%d,%s>", t, p.layout, pl.vec, epi); break;
    case V_FP8: snprintf(buf, sizeof buf, "ks_fp8_kernel<%d,%d,%d>", p.layout, pl.vec, pl.waves_m); break;
    default: snprintf(buf, sizeof buf, "?");
  }
  std::string r(buf);
  r.erase(std::remove(r.begin(), r.end(), ' '), r.end());
  return r;
}

std::string describe(const Problem& p, const Plan& pl) {
  static const char* names[] = {"generic", "valu_bsl", "valu_bsf", "direct", "staged", "?", "dma", "masked", "fp8"};
  char buf[320];
  snprintf(buf, sizeof buf,
           "variant=%d name=%s vec=%d bt=%d jg=%d unroll=%d waves_m=%d waves_n=%d lds=%d grid=%u block=%u xcd=%d "
           "rs=%d kgw=%d lch=%d nt=%d kernel=%s",
           pl.variant, (pl.variant >= 0 && pl.variant < V_COUNT) ? names[pl.variant] : "?", pl.vec, pl.bt, pl.jg,
           pl.unroll, pl.waves_m, pl.waves_n, pl.lds_bytes, pl.grid, pl.block, pl.xcd_remap, pl.rs, pl.kgw, pl.lch,
           pl.nt, kernel_name(p, pl).c_str());
  return buf;
}

constexpr size_t kWsAlign = 256;
size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Bytes of one intermediate buffer of the chain (largest intermediate width),
// or 0 if the arguments are invalid.
ks_status_t chain_check(const ks_factor_t* f, int n, int64_t batch, int dtype, size_t* per_buf) {
  if (f == nullptr || n < 1) return KS_ERR_INVALID_ARG;
  // (FP8 chains are not supported: a factor's bf16 output is not the next
  // factor's FP8 input.)
  if (dtype != KS_F32 && dtype != KS_BF16 && dtype != KS_F16) return KS_ERR_UNSUPPORTED;
  if (batch < 0) return KS_ERR_INVALID_ARG;
  int64_t widest = 0;
  for (int q = 0; q < n; ++q) {
    Dims dm;
    ks_status_t st = check_pattern(f[q].a, f[q].b, f[q].c, f[q].d, &dm);
    if (st != KS_OK) return st;
    if (q + 1 < n) {
      Dims nx;
      st = check_pattern(f[q + 1].a, f[q + 1].b, f[q + 1].c, f[q + 1].d, &nx);
      if (st != KS_OK) return st;
      if (dm.N != nx.M) return KS_ERR_DIM_MISMATCH;
      widest = std::max(widest, dm.N);  // output of factor q+1 = input of factor q
    }
  }
  int64_t elems;
  if (!mul_ok(widest, batch, &elems) || elems > kMaxElems) return KS_ERR_UNSUPPORTED;
  *per_buf = round_up((size_t)elems * (size_t)elem_size(dtype), kWsAlign);
  return KS_OK;
}

}  // namespace
}  // namespace ks

namespace ks {
// The chain driver behind ks_chain (and ks_chain_noalloc, which passes its
// fixed scratch buffer as the workspace).
void set_last_hip_error(int e) { g_last_hip_error = e; }

// The fused chain kernel (ks_chain_fused.h) takes chains of two or more
// factors whose blocks are all at most 8 x 8, or all square with one b = c
// in {16, 32, 48, 64} (the MFMA form, batch-size-first), and whose widest
// vector, for 16
// batch columns in fp32, fits the kernel's 160 KB of LDS (next to one pass's
// factor values for small blocks; in place when every factor has b == c,
// else two buffers).  Not used while a kernel variant is forced or fusion is
// switched off on this thread.  Fills the pattern part of `fc`.
bool chain_fused_plan(const ks_factor_t* f, int n, int64_t batch, int layout, int dtype, FusedChain* fc) {
  if (g_forced_variant >= 0 || g_chain_fusion == 0) return false;
  if (n < 2 || n > kFusedMaxFactors) return false;
  int64_t wmax = 0;
  bool inplace = true, small = true, square16 = true;
  for (int q = 0; q < n; ++q) {
    small = small && f[q].b <= kFusedMaxBC && f[q].c <= kFusedMaxBC;
    square16 = square16 && f[q].b == f[q].c && f[q].b == f[0].b && f[q].b % 16 == 0 && f[q].b <= kFusedMfmaMaxB;
    const int64_t N = f[q].a * f[q].c * f[q].d, M = f[q].a * f[q].b * f[q].d;
    wmax = std::max(wmax, std::max(N, M));
    inplace = inplace && f[q].b == f[q].c;
  }
  if (!small && !square16) return false;
  // The MFMA form: batch-size-first in every type; batch-size-last only in
  // fp32, with tiles of 32 columns, whose row pieces are whole 128-byte lines.
  // Narrower pieces (16-bit types, or 16 fp32 columns) are read and written
  // faster by the factor-by-factor kernels, which run along the batch.
  const bool wide_fits = wmax * (2 * kFusedCols + 4) * 4 <= kFusedMaxLds && f[0].b <= 32;
  if (!small && layout != KS_LAYOUT_BSF && !(dtype == KS_F32 && wide_fits)) return false;
  const int64_t kbuf = small ? kFusedKValues : 0;
  if (((inplace ? 1 : 2) * wmax * kFusedPitch + kbuf) * 4 > kFusedMaxLds) return false;
  if ((batch + kFusedCols - 1) / kFusedCols > 0x7fffffff) return false;
  fc->nf = n;
  fc->batch = (int)batch;
  fc->layout = layout;
  fc->width_in = (int)(f[n - 1].a * f[n - 1].c * f[n - 1].d);
  fc->width_out = (int)(f[0].a * f[0].b * f[0].d);
  fc->inplace = inplace ? 1 : 0;
  fc->buf_rows = (int)wmax;
  fc->kvec = 0;  // set at launch (chain_fused_kvec)
  fc->mfma = small ? 0 : 1;
  fc->cols = kFusedCols;
  fc->pitch = kFusedPitch;
  // MFMA form in fp32: tiles of 32 columns when they fit (batch-size-last
  // always; batch-size-first when the tile's 16-byte pieces per batch row
  // come in groups of 4, which its coalesced load and store order needs)
  if (!small && dtype == KS_F32 && wide_fits &&
      (layout != KS_LAYOUT_BSF || (fc->width_in % 16 == 0 && fc->width_out % 16 == 0))) {
    fc->cols = 2 * kFusedCols;
    fc->pitch = 2 * kFusedCols + 4;
  }
  // the dyadic butterfly of size 2^L, L = 4 .. 10: factor q of pattern
  // (2^q, 2, 2, 2^(L-1-q)) in product order
  fc->bfly = 0;
  if (small && n >= 4 && n <= 10) {
    bool bf = true;
    for (int q = 0; q < n && bf; ++q)
      bf = f[q].b == 2 && f[q].c == 2 && f[q].a == ((int64_t)1 << q) && f[q].d == ((int64_t)1 << (n - 1 - q));
    if (bf) fc->bfly = n;
  }
  for (int q = 0; q < n; ++q) {
    fc->a[q] = (int)f[q].a; fc->b[q] = (int)f[q].b; fc->c[q] = (int)f[q].c; fc->d[q] = (int)f[q].d;
    div_magic((uint32_t)f[q].d, &fc->md[q], &fc->sd[q]);
    fc->kv[q] = f[q].K_values;
  }
  if (fc->mfma) {
    // One pass per factor; the values are read straight from global memory.
    for (int q = 0; q < n; ++q) {
      const int f0 = n - 1 - q;
      fc->pf0[q] = f0;
      fc->pm[q] = 1;
      fc->pp[q] = 0;
      fc->pP[q] = 1;
      fc->pcnt[q] = fc->pk[q] = fc->a[f0] * fc->d[f0] * fc->b[f0] * fc->c[f0];
      div_magic((uint32_t)fc->d[f0], &fc->mgd[q], &fc->sgd[q]);
    }
    fc->npass = n;
    return fused_lds_bytes(*fc) <= kFusedMaxLds;
  }
  // Passes in application order (factor n-1 first): runs of square p x p
  // factors (p in {2, 4, 8}) whose strides nest (d of the next = p * d,
  // a of the previous = p * a of the next), up to 3 factors for p = 2 (one
  // for p = 4, 8); every other factor alone.
  int np = 0;
  for (int q = n - 1; q >= 0;) {
    const int p = fc->b[q];
    int m = 1;
    if (fc->b[q] == fc->c[q] && (p == 2 || p == 4 || p == 8)) {
      const int maxm = p == 2 ? 3 : 1;
      while (m < maxm && q - m >= 0) {
        const int g = q - m, prev = q - m + 1;
        if (fc->b[g] == p && fc->c[g] == p && fc->d[g] == p * fc->d[prev] && fc->a[prev] == p * fc->a[g]) ++m;
        else break;
      }
      int P = 1;
      for (int t = 0; t < m; ++t) P *= p;
      fc->pp[np] = p;
      fc->pP[np] = P;
    } else {
      fc->pp[np] = 0;
      fc->pP[np] = 1;
    }
    fc->pf0[np] = q;
    fc->pm[np] = m;
    fc->pcnt[np] = fc->a[q] * fc->d[q] * fc->b[q] * fc->c[q];
    fc->pk[np] = m * fc->pcnt[np];
    if (fc->pk[np] > kFusedKValues) return false;
    div_magic((uint32_t)fc->d[q], &fc->mgd[np], &fc->sgd[np]);
    ++np;
    q -= m;
  }
  fc->npass = np;
  return fused_lds_bytes(*fc) <= kFusedMaxLds;
}

// 16-byte vectors for the fused kernel's loads and stores: aligned buffers and
// a batch (BSL) or widths (BSF) that are whole vectors.
bool chain_fused_vec(const FusedChain& fc, int dtype, const void* X, const void* Y) {
  const int e = 16 / elem_size(dtype);
  if (!aligned16(X) || !aligned16(Y)) return false;
  if (fc.layout == BSL) return fc.batch % e == 0;
  return fc.width_in % e == 0 && fc.width_out % e == 0;
}

// Runs of 4 factor values per load: every pass's per-factor count is a
// multiple of 4 and every factor's values are aligned to 4 elements.
bool chain_fused_kvec(const FusedChain& fc, int dtype) {
  const uintptr_t al = 4 * (uintptr_t)elem_size(dtype);
  for (int q = 0; q < fc.nf; ++q)
    if (reinterpret_cast<uintptr_t>(fc.kv[q]) % al) return false;
  for (int q = 0; q < fc.npass; ++q)
    if (fc.pcnt[q] % 4) return false;
  return true;
}

ks_status_t chain_impl(const ks_factor_t* factors, int nfactors, const void* X, void* Y, int64_t batch, int layout,
                       int dtype, void* workspace, size_t workspace_bytes, void* stream) {
  size_t per = 0;
  ks_status_t st = chain_check(factors, nfactors, batch, dtype, &per);
  if (st != KS_OK) return st;
  if (layout != KS_LAYOUT_BSF && layout != KS_LAYOUT_BSL) return KS_ERR_UNSUPPORTED;
  for (int q = 0; q < nfactors; ++q)
    if (factors[q].K_values == nullptr) return KS_ERR_INVALID_ARG;
  FusedChain fc;
  const bool fused = chain_fused_plan(factors, nfactors, batch, layout, dtype, &fc);
  const size_t need = (fused || nfactors <= 1) ? 0 : (nfactors == 2 ? per : 2 * per);
  if (batch == 0) return KS_OK;
  if (X == nullptr || Y == nullptr) return KS_ERR_INVALID_ARG;
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return KS_ERR_WORKSPACE;
  const int s = elem_size(dtype);
  Dims first, last;
  check_pattern(factors[0].a, factors[0].b, factors[0].c, factors[0].d, &first);
  check_pattern(factors[nfactors - 1].a, factors[nfactors - 1].b, factors[nfactors - 1].c,
                factors[nfactors - 1].d, &last);
  int64_t xe, ye;
  if (!mul_ok(batch, last.N, &xe) || !mul_ok(batch, first.M, &ye) || xe > kMaxElems || ye > kMaxElems)
    return KS_ERR_UNSUPPORTED;
  if (overlaps(X, xe * s, Y, ye * s)) return KS_ERR_ALIAS;
  if (need > 0 && (overlaps(workspace, (int64_t)need, X, xe * s) || overlaps(workspace, (int64_t)need, Y, ye * s)))
    return KS_ERR_ALIAS;
  if (fused) {
    fc.x = X;
    fc.y = Y;
    fc.kvec = chain_fused_kvec(fc, dtype) ? 1 : 0;
    const hipError_t e = launch_chain_fused(fc, dtype, chain_fused_vec(fc, dtype, X, Y), static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
      g_last_hip_error = (int)e;
      return KS_ERR_HIP;
    }
    return KS_OK;
  }
  // Validate every step before enqueueing anything.
  char* ws = static_cast<char*>(workspace);
  void* bufs[2] = {ws, ws + per};
  Problem steps[64];
  Problem* pv = nfactors <= 64 ? steps : new Problem[nfactors];
  const void* in = X;
  int which = 0;
  for (int q = nfactors - 1; q >= 0; --q) {
    void* out = (q == 0) ? Y : bufs[which];
    bool empty = false;
    st = validate(factors[q].a, factors[q].b, factors[q].c, factors[q].d, factors[q].K_values, in, out, batch, layout,
                  dtype, &pv[q], &empty);
    if (st != KS_OK) break;
    in = out;
    which ^= 1;
  }
  if (st == KS_OK) {
    for (int q = nfactors - 1; q >= 0 && st == KS_OK; --q) st = run_one(pv[q], static_cast<hipStream_t>(stream));
  }
  if (pv != steps) delete[] pv;
  return st;
}
}  // namespace ks

using namespace ks;

extern "C" {

ks_status_t ks_matmul(int64_t a, int64_t b, int64_t c, int64_t d, const void* K_values, const void* X, void* Y,
                      int64_t batch, int layout, int dtype, void* stream) {
  Problem p;
  bool empty = false;
  ks_status_t st = validate(a, b, c, d, K_values, X, Y, batch, layout, dtype, &p, &empty);
  if (st != KS_OK || empty) return st;
  return run_one(p, static_cast<hipStream_t>(stream));
}

ks_status_t ks_matmul_bias_act(int64_t a, int64_t b, int64_t c, int64_t d, const void* K_values, const void* bias,
                               int act, const void* X, void* Y, int64_t batch, int layout, int dtype, void* stream) {
  Problem p;
  bool empty = false;
  ks_status_t st = validate(a, b, c, d, K_values, X, Y, batch, layout, dtype, &p, &empty);
  if (st != KS_OK) return st;
  if (act != KS_ACT_NONE && act != KS_ACT_GELU) return KS_ERR_UNSUPPORTED;
  if (empty) return KS_OK;
  if (bias != nullptr && overlaps(bias, (int64_t)p.M * out_size(dtype), Y, (int64_t)p.batch * p.M * out_size(dtype)))
    return KS_ERR_ALIAS;
  p.bias = bias;
  p.act = act;
  return run_one(p, static_cast<hipStream_t>(stream));
}

size_t ks_chain_workspace_bytes(const ks_factor_t* factors, int nfactors, int64_t batch, int dtype) {
  size_t per = 0;
  if (chain_check(factors, nfactors, batch, dtype, &per) != KS_OK) return 0;
  if (nfactors <= 1) return 0;
  FusedChain fc;
  // the workspace of the layout that needs one (the size does not depend on the layout)
  if (chain_fused_plan(factors, nfactors, batch, KS_LAYOUT_BSL, dtype, &fc) &&
      chain_fused_plan(factors, nfactors, batch, KS_LAYOUT_BSF, dtype, &fc))
    return 0;
  return nfactors == 2 ? per : 2 * per;
}

void ks_force_chain_fusion(int mode) { g_chain_fusion = mode < 0 ? -1 : (mode == 0 ? 0 : -1); }

ks_status_t ks_chain_describe(const ks_factor_t* factors, int nfactors, int64_t batch, int layout, int dtype,
                              char* buf, size_t len) {
  if (buf == nullptr || len == 0) return KS_ERR_INVALID_ARG;
  buf[0] = 0;
  size_t per = 0;
  ks_status_t st = chain_check(factors, nfactors, batch, dtype, &per);
  if (st != KS_OK) return st;
  if (layout != KS_LAYOUT_BSF && layout != KS_LAYOUT_BSL) return KS_ERR_UNSUPPORTED;
  FusedChain fc;
  if (chain_fused_plan(factors, nfactors, batch, layout, dtype, &fc)) {
    std::string passes;
    for (int q = 0; q < fc.npass; ++q) {
      char pb[32];
      snprintf(pb, sizeof pb, "%s%d", q ? "," : "", fc.pp[q] ? fc.pP[q] : -fc.b[fc.pf0[q]]);
      passes += pb;
    }
    if (fc.bfly) passes = std::to_string(1 << bfly_la(fc.bfly)) + "," + std::to_string(1 << (fc.bfly - bfly_la(fc.bfly)));
    snprintf(buf, len, "fused%s factors=%d passes=%d groups=%s inplace=%d lds=%d grid=%lld block=%d cols=%d",
             fc.mfma ? "-mfma" : (fc.bfly ? "-bfly" : ""), fc.nf, fc.bfly ? 2 : fc.npass, passes.c_str(), fc.inplace,
             fused_lds_bytes(fc), (long long)((batch + fc.cols - 1) / fc.cols), kFusedThreads, fc.cols);
  } else {
    snprintf(buf, len, "unfused factors=%d workspace=%zu", nfactors, nfactors <= 1 ? (size_t)0 : (nfactors == 2 ? per : 2 * per));
  }
  return KS_OK;
}

ks_status_t ks_chain(const ks_factor_t* factors, int nfactors, const void* X, void* Y, int64_t batch, int layout,
                     int dtype, void* workspace, size_t workspace_bytes, void* stream) {
  return ks::chain_impl(factors, nfactors, X, Y, batch, layout, dtype, workspace, workspace_bytes, stream);
}

const char* ks_status_string(int status) {
  switch (status) {
    case KS_OK: return "KS_OK";
    case KS_ERR_INVALID_PATTERN: return "KS_ERR_INVALID_PATTERN: a, b, c and d must be >= 1 and their products fit int64";
    case KS_ERR_INVALID_ARG: return "KS_ERR_INVALID_ARG: null pointer, negative batch or bad factor count";
    case KS_ERR_DIM_MISMATCH: return "KS_ERR_DIM_MISMATCH: chain factors do not compose (a*c*d of one != a*b*d of next)";
    case KS_ERR_ALIAS: return "KS_ERR_ALIAS: output overlaps an input or the workspace";
    case KS_ERR_UNSUPPORTED: return "KS_ERR_UNSUPPORTED: unsupported dtype/layout/size, or forced variant cannot run";
    case KS_ERR_WORKSPACE: return "KS_ERR_WORKSPACE: chain workspace missing or too small";
    case KS_ERR_HIP: return "KS_ERR_HIP: the HIP runtime reported an error";
    case KS_ERR_SCRATCH_LIMIT:
      return "KS_ERR_SCRATCH_LIMIT: the chain's intermediates exceed the fixed scratch array of ks_chain_noalloc";
    default: return "unknown ks_status_t";
  }
}

int ks_last_hip_error(void) { return g_last_hip_error; }

ks_status_t ks_plan_describe(int64_t a, int64_t b, int64_t c, int64_t d, int64_t batch, int layout, int dtype,
                             char* buf, size_t len) {
  if (buf == nullptr || len == 0) return KS_ERR_INVALID_ARG;
  buf[0] = 0;
  // Validate with stand-in, 256-byte-aligned, non-overlapping addresses: the plan
  // depends on pointer alignment only, and aligned buffers are the common case.
  Dims dm;
  ks_status_t st = check_pattern(a, b, c, d, &dm);
  if (st != KS_OK) return st;
  const uintptr_t base = uintptr_t(1) << 44;
  const uintptr_t span = uintptr_t(1) << 40;
  Problem p;
  bool empty = false;
  st = validate(a, b, c, d, reinterpret_cast<const void*>(base), reinterpret_cast<const void*>(base + span),
                reinterpret_cast<void*>(base + 2 * span), batch, layout, dtype, &p, &empty);
  if (st != KS_OK) return st;
  if (empty) {
    snprintf(buf, len, "empty");
    return KS_OK;
  }
  Plan pl;
  if (!get_plan(p, true, &pl)) return KS_ERR_UNSUPPORTED;
  snprintf(buf, len, "%s", describe(p, pl).c_str());
  return KS_OK;
}

void ks_force_variant(int variant) { g_forced_variant = variant < 0 ? -1 : variant; }

}  // extern "C"

namespace ks {
// Plan for stand-in aligned buffers (used by the host-side verifier).  Returns
// false (with *st set) when there is nothing to launch or no plan.
bool plan_for_verify(int64_t a, int64_t b, int64_t c, int64_t d, int64_t batch, int layout, int dtype, Problem* p,
                     Plan* pl, ks_status_t* st) {
  const uintptr_t base = uintptr_t(1) << 44;
  const uintptr_t span = uintptr_t(1) << 40;
  bool empty = false;
  *st = validate(a, b, c, d, reinterpret_cast<const void*>(base), reinterpret_cast<const void*>(base + span),
                 reinterpret_cast<void*>(base + 2 * span), batch, layout, dtype, p, &empty);
  if (*st != KS_OK || empty) return false;
  if (!get_plan(*p, true, pl)) {
    *st = KS_ERR_UNSUPPORTED;
    return false;
  }
  return true;
}
}  // namespace ks
