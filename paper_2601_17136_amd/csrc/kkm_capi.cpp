// Host side of the engine: the C ABI declared in include/kkm.h.
//
// A context owns every device buffer.  kkm_build_kernel stages the points and
// (resident and packed modes) builds K; kkm_iterate runs the loop body of
// Alg. 1 with one process: scatter -> SpMM -> reduce -> assign per update,
// enqueued back to back on the context's stream with no host round trip
// unless a stop test needs one.  Argument checks run before any HIP call.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kkm.h"
#include "kkm_internal.h"

using namespace kkm;

// Device scratch of kkm_iterate_noalloc: one copy per GPU, held until the
// process ends.  Host code never passes this name to a kernel or a copy (on
// the host it is a stand-in, not a device address); it uses the address
// hipGetSymbolAddress returns for the current device, looked up once per
// device by kkm_create.
static __device__ __align__(256) unsigned char scratch[KKM_NOALLOC_SCRATCH_BYTES];

namespace {

std::mutex g_scratch_mu;
std::vector<void*> g_scratch_ptr;  // by device ordinal; null until looked up

// The device address of `scratch` on device dev (current), looked up once.
hipError_t scratch_address(int dev, void** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if ((int)g_scratch_ptr.size() <= dev) g_scratch_ptr.resize(dev + 1, nullptr);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}


struct TimedLaunch {
  int phase;
  hipEvent_t start, stop;
};

struct Alloc {
  void* p;
  size_t bytes;
};

thread_local std::string g_noctx_err;
thread_local std::string g_noctx_warn;  // last warning of kkm_check_build_args on this thread

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// Error estimate for the Gaussian expansion s = |x|^2 + |y|^2 - 2 x.y in fp32:
// |err(s)| ~ kFixAcc * 2^-24 * (|x|^2 + |y|^2), and the entry moves by
// gamma * err(s) * K.  Entries where that exceeds kFixTol are recomputed.
constexpr float kFixAcc = 8.0f;
constexpr float kFixTol = 2.0e-6f;

struct Sizes {
  int64_t n, n_pad, ld, nblk;
  int d_pad, nstripes;
};

// Packed K keeps whole column tiles, so its rows run to n_pad.
Sizes sizes_for(int64_t n, int32_t d, int mode) {
  Sizes s;
  s.n = n;
  s.n_pad = round_up(n, kTile);
  s.ld = mode == KKM_MODE_PACKED ? s.n_pad : round_up(n, 64);
  s.d_pad = (int)round_up(d, 8);  // the K-build mainloop takes a last chunk of 8
  s.nblk = (n + kBlk - 1) / kBlk;
  s.nstripes = (int)((s.ld + kStripe - 1) / kStripe);
  return s;
}

// staged points, their norms, diag K, and the largest norm of each 128-point block
size_t staged_bytes(const Sizes& s) {
  return (size_t)s.n_pad * s.d_pad * 4 + (size_t)s.n_pad * 4 + (size_t)s.n * 4 + (size_t)(s.n_pad / kTile) * 4 + 64;
}
// bytes of one stored entry of K
size_t k_elem(int storage) { return storage == KKM_STORE_F16 ? 2 : 4; }
size_t k_bytes(const Sizes& s, int mode, int storage) {
  if (mode == KKM_MODE_PACKED) return (size_t)packed_floats(s.n, s.ld) * k_elem(storage);
  return mode == KKM_MODE_RESIDENT ? (size_t)s.n * (size_t)s.ld * k_elem(storage) : 0;
}
// The linear and polynomial kernels keep a bound per row of |K(i, .)| where
// K is stored in binary16 (the stored values are K / bound) or packed (the
// packed SpMM's column side scales each row by the power of two at or above
// its bound).  The Gaussian's entries lie in [0, 1] and need none.
bool row_scaled(int mode, int storage, int kind) {
  return kind != KKM_GAUSS &&
         (mode == KKM_MODE_PACKED || (storage == KKM_STORE_F16 && mode == KKM_MODE_RESIDENT));
}
int chunk_len_for(const Sizes& s, int mode) { return mode == KKM_MODE_PACKED ? sym_chunk_for(s.n) : kChunk; }
int64_t qmax_for(const Sizes& s, int k, int mode) {
  const int64_t c = chunk_len_for(s, mode);
  return (s.n + c - 1) / c + k;
}
int nseg_for(const Sizes& s, int k) {
  const int bseg = sym_seg_for(s.n, k);
  return (int)((s.n_pad / kTile + bseg - 1) / bseg);
}
// self-term partials per cluster: one per stripe of the mode's reduction
int nzpart_for(const Sizes& s, int mode) {
  return mode == KKM_MODE_PACKED ? (int)((s.ld + kSymRedStripe - 1) / kSymRedStripe) : s.nstripes;
}

size_t ws_bytes(const Sizes& s, int k, int mode) {
  const int64_t qmax = qmax_for(s, k, mode);
  size_t b = 0;
  b += (size_t)k * s.ld * 4;              // Et
  if (mode == KKM_MODE_RESIDENT || mode == KKM_MODE_PACKED) {
    b += (size_t)qmax * s.ld * 4;         // P: chunk partials
  }
  if (mode == KKM_MODE_PACKED) {
    b += (size_t)nseg_for(s, k) * k * qmax * chunk_len_for(s, mode) * 4;  // Ecp: column-side partials
    b += (size_t)k * s.n * 4;                // Ecol
    b += (size_t)qmax * 4;                   // chunk start columns
    b += (size_t)qmax * chunk_len_for(s, mode) * 4;  // chunk-major member table
    b += (size_t)(s.n_pad / kTile) * ((k + 15) / 16) * 64 * 4;  // one-hot bits per column tile
    b += (size_t)kTile * 4;                  // zero page
  } else if (mode == KKM_MODE_ONTHEFLY) {
    b += (size_t)s.n_pad * s.d_pad * 4;   // sorted points
    b += (size_t)s.n_pad * 8;             // their norms and cluster ids
    const size_t halves = (size_t)onthefly_halves(s.d_pad);
    b += halves * onthefly_segments(s.n) * k * s.ld * 4;  // row-side segment partials
    b += halves * onthefly_cpart_floats(s.n, k) * 4;      // column-side partials
    b += (size_t)(s.n_pad / kTile) * 20;                 // per-block tables
  }
  b += (size_t)k * nzpart_for(s, mode) * 8;  // zpart
  b += (size_t)2 * k * s.nblk * 4;        // hist, base
  b += (size_t)2 * (k + 1) * 4;           // off, qfirst
  b += (size_t)3 * qmax * 4 + 4;          // chunk table
  b += (size_t)4 * s.n * 4;               // perm, pos, two id buffers
  b += (size_t)2 * k * 4 + 64;            // counts, status
  return b + 40 * 256;                    // alignment slack
}

}  // namespace

struct kkm_ctx {
  hipStream_t stream = nullptr;
  int device = 0;
  size_t budget = 0, held = 0;
  std::string err;
  std::string warn;  // warning of the last build ("" if none)

  bool built = false;
  // A block of K (one GPU's share): rows [pr0, pr1) and columns [pc0, pc1);
  // pc1 = 0 for the full K.  A panel is the block of all rows.
  int64_t pr0 = 0, pr1 = 0, pc0 = 0, pc1 = 0;
  bool panel_e = false;       // the panel's E^T and sizes are current (kkm_panel_spmm ran)
  Sizes sz{};                 // the problem: n points (staging, norms, diag K)
  Sizes wsz{};                // the stored K and the scratch: sz, or a block's rows as n
  int d = 0, kind = 0, mode = 0;
  kkm_params params{};
  KappaParams kp{};
  float *Xp = nullptr, *nrm = nullptr, *diagK = nullptr;
  float* bmax = nullptr;      // largest squared norm of each 128-point block of the staged points
  void* K = nullptr;          // fp32 or binary16 entries (storage)
  int storage = KKM_STORE_F32;
  float* kw = nullptr;        // binary16 row scales (linear, polynomial), else null
  double* trK = nullptr;
  unsigned* maxnrm = nullptr;  // bits of the largest squared norm (next to tr K)
  int2* fix_list = nullptr;
  unsigned long long* fix_count = nullptr;  // kFixSegs counters
  long long fix_cap = 0;                    // entries in all segments together
  int64_t fixups = 0;
  std::vector<Alloc> build_allocs;

  int k_ws = 0, iter_ws = 0;
  IterBufs ib{};
  float *Xs = nullptr, *nrm_s = nullptr, *Epart = nullptr, *Cpart = nullptr;  // on-the-fly scratch
  int* cs = nullptr;
  OtfTables otb{};
  const int* epos = nullptr;  // column order of E^T after the last update (null: identity)
  int* counts[2] = {nullptr, nullptr};
  int* clbuf[2] = {nullptr, nullptr};
  std::vector<Alloc> ws_allocs;
  int* changed = nullptr;
  double* obj = nullptr;
  std::vector<Alloc> hist_allocs;

  // K-means++ seeding scratch (first use after a build): n floats kd, D,
  // best, n ints bestc, per-block fp64 sums, KKM_MAX_K center indices
  std::vector<Alloc> seed_allocs;
  float *sd_kd = nullptr, *sd_D = nullptr, *sd_best = nullptr;
  int *sd_bestc = nullptr, *sd_centers = nullptr;
  double* sd_bsum = nullptr;

  void* scratch = nullptr;  // this device's static scratch (kkm_iterate_noalloc)

  int32_t timing = 0;  // mask of timed phases
  std::vector<TimedLaunch> pending;
  std::vector<hipEvent_t> pool;
  kkm_timing tacc{};
};

namespace {

int fail(kkm_ctx* c, int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf;
  else g_noctx_err = buf;
  return code;
}

int hip_fail(kkm_ctx* c, hipError_t e, const char* what) {
  return fail(c, KKM_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(c, expr, what)                    \
  do {                                            \
    hipError_t e_ = (expr);                       \
    if (e_ != hipSuccess) return hip_fail(c, e_, what); \
  } while (0)

// K, and the iteration scratch the SpMM reads its chunk tables from and
// writes its partial sums into, are allocated as physically contiguous memory
// when K is at least this large (hipMalloc is the fallback).  With K of 7 GB
// and more, the packed SpMM measured 3.6% faster (60000 points) and 6% faster
// (200000 points) with a contiguous scratch than with one from hipMalloc, on
// the same K, and the full-K SpMM 0.6-2%; with K of 1.6 GB and less it
// measured 0.5-7% slower, so small problems keep hipMalloc.
constexpr size_t kContiguousFromK = (size_t)4 << 30;

int dalloc(kkm_ctx* c, void** p, size_t bytes, std::vector<Alloc>& owner, const char* what,
           bool contiguous = false) {
  bytes = std::max<size_t>(bytes, 256);
  if (c->held + bytes > c->budget)
    return fail(c, KKM_ERR_OOM, "%s needs %zu bytes; %zu of the %zu-byte budget already held", what,
                bytes, c->held, c->budget);
  hipError_t e = hipErrorOutOfMemory;
  if (contiguous) {
    e = hipExtMallocWithFlags(p, bytes, hipDeviceMallocContiguous);
    if (e != hipSuccess) (void)hipGetLastError();
  }
  if (e != hipSuccess) e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    *p = nullptr;
    return fail(c, KKM_ERR_OOM, "hipMalloc(%zu) for %s: %s", bytes, what, hipGetErrorString(e));
  }
  owner.push_back({*p, bytes});
  c->held += bytes;
  return KKM_OK;
}

void release(kkm_ctx* c, std::vector<Alloc>& owner) {
  for (const Alloc& a : owner) {
    (void)hipFree(a.p);
    c->held -= std::min(c->held, a.bytes);
  }
  owner.clear();
}

hipEvent_t take_event(kkm_ctx* c) {
  if (!c->pool.empty()) {
    hipEvent_t e = c->pool.back();
    c->pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <class F>
int run(kkm_ctx* c, int phase, const char* what, F&& f) {
  hipEvent_t a = nullptr, b = nullptr;
  const bool timed = (c->timing >> phase) & 1;
  if (timed) {
    a = take_event(c);
    b = take_event(c);
    if (a) (void)hipEventRecord(a, c->stream);
  }
  hipError_t e = f();
  if (timed && a && b) {
    (void)hipEventRecord(b, c->stream);
    c->pending.push_back({phase, a, b});
  }
  if (e != hipSuccess) return hip_fail(c, e, what);
  return KKM_OK;
}

void collect_timing(kkm_ctx* c) {
  for (auto& t : c->pending) {
    float ms = 0.f;
    if (hipEventSynchronize(t.stop) == hipSuccess && hipEventElapsedTime(&ms, t.start, t.stop) == hipSuccess) {
      c->tacc.ms[t.phase] += ms;
      c->tacc.launches[t.phase] += 1;
    }
    c->pool.push_back(t.start);
    c->pool.push_back(t.stop);
  }
  c->pending.clear();
}

void free_ws(kkm_ctx* c) {
  release(c, c->ws_allocs);
  c->k_ws = 0;
  c->ib = IterBufs{};
  c->Xs = c->nrm_s = c->Epart = c->Cpart = nullptr;
  c->cs = nullptr;
  c->otb = OtfTables{};
}

void free_hist(kkm_ctx* c) {
  release(c, c->hist_allocs);
  c->iter_ws = 0;
  c->changed = nullptr;
  c->obj = nullptr;
}

void free_seed(kkm_ctx* c) {
  release(c, c->seed_allocs);
  c->sd_kd = c->sd_D = c->sd_best = nullptr;
  c->sd_bestc = c->sd_centers = nullptr;
  c->sd_bsum = nullptr;
}

void free_build(kkm_ctx* c) {
  free_ws(c);
  free_hist(c);
  free_seed(c);
  release(c, c->build_allocs);
  c->Xp = c->nrm = c->diagK = c->bmax = nullptr;
  c->K = nullptr;
  c->kw = nullptr;
  c->trK = nullptr;
  c->fix_list = nullptr;
  c->fix_count = nullptr;
  c->fix_cap = 0;
  c->built = false;
  c->pr0 = c->pr1 = c->pc0 = c->pc1 = 0;
  c->panel_e = false;
}

// Lay the per-update scratch for k clusters out over base (ws_bytes of it)
// and clear what must start at zero.
int carve_from(kkm_ctx* c, int k, void* base) {
  const Sizes& s = c->wsz;
  int rc;
  char* p = (char*)base;
  auto take = [&](size_t bytes) {
    char* r = p;
    p += (bytes + 255) / 256 * 256;
    return (void*)r;
  };
  IterBufs& b = c->ib;
  b = IterBufs{};
  b.n = s.n;
  b.ld = s.ld;
  b.k = k;
  b.nblk = (int)s.nblk;
  b.nstripes = s.nstripes;
  b.nzpart = nzpart_for(s, c->mode);
  const int64_t qmax = qmax_for(s, k, c->mode);
  b.qmax = (int)qmax;
  b.chunk_len = chunk_len_for(s, c->mode);
  b.diagK = c->diagK;
  b.col0 = c->pc1 > 0 ? c->pc0 : 0;
  b.ncol = c->pc1 > 0 ? c->pc1 - c->pc0 : s.n;
  b.trK = c->trK;
  b.kf16 = c->storage == KKM_STORE_F16;
  b.kw = c->kw;
  b.Et = (float*)take((size_t)k * s.ld * 4);
  if (c->mode == KKM_MODE_RESIDENT || c->mode == KKM_MODE_PACKED) {
    b.P = (float*)take((size_t)qmax * s.ld * 4);
  }
  if (c->mode == KKM_MODE_PACKED) {
    b.nt = (int)(s.n_pad / kTile);
    b.bseg = sym_seg_for(s.n, k);
    b.nseg = nseg_for(s, k);
    b.Ecp = (float*)take((size_t)b.nseg * k * qmax * b.chunk_len * 4);
    b.Ecol = (float*)take((size_t)k * s.n * 4);
    b.chunk_c0 = (int*)take((size_t)qmax * 4);
    b.nlb = (k + 15) / 16;
    b.crow = (int*)take((size_t)qmax * b.chunk_len * 4);
    b.mskg = (unsigned*)take((size_t)b.nt * b.nlb * 64 * 4);
    float* zero = (float*)take((size_t)kTile * 4);
    b.zero = zero;
    rc = run(c, KKM_PHASE_OTHER, "zero page", [&] { return launch_zero_ints((int*)zero, kTile, c->stream); });
    if (rc) return rc;
  } else if (c->mode == KKM_MODE_ONTHEFLY) {
    c->Xs = (float*)take((size_t)s.n_pad * s.d_pad * 4);
    c->nrm_s = (float*)take((size_t)s.n_pad * 4);
    c->cs = (int*)take((size_t)s.n_pad * 4);
    const size_t halves = (size_t)onthefly_halves(s.d_pad);
    c->Epart = (float*)take(halves * onthefly_segments(s.n) * k * s.ld * 4);
    c->Cpart = (float*)take(halves * onthefly_cpart_floats(s.n, k) * 4);
    const size_t nt = (size_t)(s.n_pad / kTile);
    c->otb.cA = (int*)take(nt * 4);
    c->otb.nruns = (int*)take(nt * 4);
    c->otb.cbase = (int64_t*)take(nt * 8);
    c->otb.bmax = (float*)take(nt * 4);
  }
  b.zpart = (double*)take((size_t)k * b.nzpart * 8);
  b.hist = (int*)take((size_t)k * s.nblk * 4);
  b.base = (int*)take((size_t)k * s.nblk * 4);
  b.off = (int*)take((size_t)(k + 1) * 4);
  b.qfirst = (int*)take((size_t)(k + 1) * 4);
  b.chunk_j = (int*)take((size_t)qmax * 4);
  b.chunk_p0 = (int*)take((size_t)qmax * 4);
  b.chunk_p1 = (int*)take((size_t)qmax * 4);
  b.nchunks = (int*)take(4);
  b.perm = (int*)take((size_t)s.n * 4);
  b.pos = (int*)take((size_t)s.n * 4);
  c->clbuf[0] = (int*)take((size_t)s.n * 4);
  c->clbuf[1] = (int*)take((size_t)s.n * 4);
  c->counts[0] = (int*)take((size_t)k * 4);
  c->counts[1] = (int*)take((size_t)k * 4);
  b.status = (int*)take(4);
  c->k_ws = k;
  return KKM_OK;
}

// The context's per-update scratch pointers, set aside while
// kkm_iterate_noalloc lays its own out over the static scratch.
struct SavedWs {
  IterBufs ib;
  int k_ws, iter_ws;
  float *Xs, *nrm_s, *Epart, *Cpart;
  int* cs;
  OtfTables otb;
  const int* epos;
  int *counts[2], *clbuf[2], *changed;
  double* obj;
};

SavedWs save_ws(const kkm_ctx* c) {
  return SavedWs{c->ib, c->k_ws, c->iter_ws, c->Xs, c->nrm_s, c->Epart, c->Cpart, c->cs, c->otb, c->epos,
                 {c->counts[0], c->counts[1]}, {c->clbuf[0], c->clbuf[1]}, c->changed, c->obj};
}

void restore_ws(kkm_ctx* c, const SavedWs& v) {
  c->ib = v.ib;
  c->k_ws = v.k_ws;
  c->iter_ws = v.iter_ws;
  c->Xs = v.Xs;
  c->nrm_s = v.nrm_s;
  c->Epart = v.Epart;
  c->Cpart = v.Cpart;
  c->cs = v.cs;
  c->otb = v.otb;
  c->epos = v.epos;
  c->counts[0] = v.counts[0];
  c->counts[1] = v.counts[1];
  c->clbuf[0] = v.clbuf[0];
  c->clbuf[1] = v.clbuf[1];
  c->changed = v.changed;
  c->obj = v.obj;
}

// Frees the Gaussian fix-up list of a finished build, after reading its
// counts (the one synchronisation this adds): a budget sized by kkm_plan
// (K, staged points, iteration scratch) has no room for both.
int release_fix_list(kkm_ctx* c) {
  if (!c->fix_list) return KKM_OK;
  if (c->fixups < 0) {
    unsigned long long cnt[kFixSegs] = {0};
    HIP_TRY(c, hipMemcpyAsync(cnt, c->fix_count, sizeof cnt, hipMemcpyDeviceToHost, c->stream), "read fix-up counts");
    HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
    int64_t tot = 0;
    for (int q = 0; q < kFixSegs; ++q) tot += (int64_t)cnt[q];
    c->fixups = tot;
  }
  std::vector<Alloc>& v = c->build_allocs;
  for (size_t i = 0; i < v.size(); ++i)
    if (v[i].p == (void*)c->fix_list) {
      (void)hipFree(v[i].p);
      c->held -= std::min(c->held, v[i].bytes);
      v.erase(v.begin() + (ptrdiff_t)i);
      break;
    }
  c->fix_list = nullptr;
  c->fix_count = nullptr;
  return KKM_OK;
}

// Allocate one block and carve it (keeps the accounting to one number).
int carve_ws(kkm_ctx* c, int k) {
  void* base = nullptr;
  int rc = dalloc(c, &base, ws_bytes(c->wsz, k, c->mode), c->ws_allocs, "iteration scratch",
                  k_bytes(c->wsz, c->mode, c->storage) >= kContiguousFromK);
  if (rc) return rc;
  return carve_from(c, k, base);
}

int ensure_ws(kkm_ctx* c, int k, int iters) {
  if (c->k_ws != k) {
    free_ws(c);
    const size_t need = ws_bytes(c->wsz, k, c->mode) + (size_t)std::max(iters, 64) * 12 + 512;
    if (c->held + need > c->budget) {
      int rc = release_fix_list(c);
      if (rc) return rc;
    }
    int rc = carve_ws(c, k);
    if (rc) return rc;
  }
  // A rebuild of the same shape keeps the scratch, but a panel or block of
  // that shape may sit at other columns of K: the fields that locate it (and
  // the build's buffers) are refreshed on every call.
  IterBufs& b = c->ib;
  b.col0 = c->pc1 > 0 ? c->pc0 : 0;
  b.ncol = c->pc1 > 0 ? c->pc1 - c->pc0 : c->wsz.n;
  b.diagK = c->diagK;
  b.trK = c->trK;
  b.kw = c->kw;
  b.kf16 = c->storage == KKM_STORE_F16;
  if (c->iter_ws < iters || !c->obj) {
    free_hist(c);
    int cap = std::max(iters, 64);
    void* p = nullptr;
    int rc = dalloc(c, &p, (size_t)cap * 12 + 512, c->hist_allocs, "objective history");
    if (rc) return rc;
    c->obj = (double*)p;
    c->changed = (int*)((char*)p + (size_t)cap * 8);
    c->iter_ws = cap;
  }
  return KKM_OK;
}

// Validate ids, count cluster sizes and per-block histograms (asynchronous;
// the status word is read at the caller's final synchronisation).
int label_pass(kkm_ctx* c, const int32_t* V) {
  IterBufs& b = c->ib;
  int rc;
  if ((rc = run(c, KKM_PHASE_LABELS, "zero", [&] { return launch_zero_ints(c->counts[0], b.k, c->stream); })))
    return rc;
  if ((rc = run(c, KKM_PHASE_LABELS, "zero", [&] { return launch_zero_ints(b.status, 1, c->stream); })))
    return rc;
  return run(c, KKM_PHASE_LABELS, "assign(labels)", [&] {
    return launch_assign(0, b, nullptr, V, nullptr, nullptr, c->counts[0], nullptr, nullptr,
                         nullptr, nullptr, c->stream);
  });
}

int status_error(kkm_ctx* c, int status) {
  if (status & 1) return fail(c, KKM_ERR_DEVICE_DATA, "a cluster id is outside [0, %d)", c->ib.k);
  return KKM_OK;
}

// One update: ids cur (sizes in counts[t&1]) -> ids nxt (sizes in counts[(t+1)&1]).
int one_update(kkm_ctx* c, int t, const int* cur, int* nxt, float* z_out, float* D_out) {
  IterBufs& b = c->ib;
  int* cin = c->counts[t & 1];
  int* cout = c->counts[(t + 1) & 1];
  int rc;
  if ((rc = run(c, KKM_PHASE_SCATTER, "scatter", [&] {
         return launch_scatter(b, cur, cin, cout, c->changed + t, c->stream);
       })))
    return rc;
  const int* pos = nullptr;
  if (c->mode == KKM_MODE_RESIDENT) {
    if ((rc = run(c, KKM_PHASE_SPMM, "spmm_onehot", [&] { return launch_spmm_onehot(c->K, b, c->stream); })))
      return rc;
    if ((rc = run(c, KKM_PHASE_REDUCE, "spmm_reduce", [&] { return launch_spmm_reduce(b, cur, c->stream); })))
      return rc;
  } else if (c->mode == KKM_MODE_PACKED) {
    if ((rc = run(c, KKM_PHASE_SPMM, "spmm_sym", [&] { return launch_spmm_sym(c->K, b, c->stream); })))
      return rc;
    if ((rc = run(c, KKM_PHASE_REDUCE, "ecol_sum", [&] { return launch_ecol_sum(b, c->stream); })))
      return rc;
    if ((rc = run(c, KKM_PHASE_REDUCE, "spmm_reduce_sym", [&] { return launch_spmm_reduce_sym(b, cur, c->stream); })))
      return rc;
  } else {
    const Sizes& s = c->sz;
    if ((rc = run(c, KKM_PHASE_OTHER, "gather_sorted", [&] {
           return launch_gather_sorted(c->Xp, c->nrm, b, cur, s.n_pad, s.d_pad, c->Xs, c->nrm_s, c->cs, c->stream);
         })))
      return rc;
    if ((rc = run(c, KKM_PHASE_ONTHEFLY, "onthefly", [&] {
           return launch_onthefly(c->Xs, c->nrm_s, c->cs, c->maxnrm, b, s.d_pad, c->kp, c->otb, c->Epart,
                                  c->Cpart, c->stream);
         })))
      return rc;
    if ((rc = run(c, KKM_PHASE_REDUCE, "onthefly_reduce", [&] {
           return launch_onthefly_reduce(b, c->Epart, c->Cpart, c->cs, c->otb, s.d_pad, c->stream);
         })))
      return rc;
    pos = b.pos;
  }
  c->epos = pos;
  return run(c, KKM_PHASE_ASSIGN, "assign", [&] {
    return launch_assign(1, b, cin, cur, pos, nxt, cout, c->changed + t, c->obj + t, z_out, D_out, c->stream);
  });
}

int check_ready(kkm_ctx* c, int32_t k, int32_t max_iter) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!c->built) return fail(c, KKM_ERR_STATE, "no kernel matrix built on this context");
  if (c->pc1 > 0) return fail(c, KKM_ERR_STATE, "the context holds a block of K; use the panel or block calls");
  if (kkm_check_iterate_args(c->sz.n, k, max_iter) != KKM_OK) return fail(c, KKM_ERR_ARG, "%s", g_noctx_err.c_str());
  if (c->mode == KKM_MODE_PACKED && k > KKM_PACKED_MAX_K)
    return fail(c, KKM_ERR_ARG, "k=%d exceeds %d, the most the packed storage handles; build RESIDENT or ONTHEFLY",
                k, KKM_PACKED_MAX_K);
  return KKM_OK;
}

// The mode AUTO resolves to, and the device bytes of a mode.  k_known: k is
// the cluster count the loop will run with; otherwise (a build without a
// hint) k only sizes the scratch and the mode is picked without it.
//   AUTO with k known: PACKED when k <= KKM_PACKED_FAST_K and it fits (it
//   streams half the bytes per update, and its per-label column side, on the
//   binary16 matrix cores, stays below the HBM time up to that many
//   labels); else RESIDENT when it fits; else ONTHEFLY.
//   AUTO with k unknown: RESIDENT, else PACKED, else ONTHEFLY, whichever
//   fits first.
// ONTHEFLY is picked only when no stored K fits: at every width measured
// (d >= 54) a stored K is at least as fast per update.  kind sizes the row
// bounds the linear and polynomial kernels keep.
int plan_impl(int64_t n, int32_t d, int32_t k, bool k_known, int32_t kind, size_t mem_budget,
              int32_t requested_mode, int32_t storage, int32_t* mode_out, size_t* bytes_out) {
  if (n < 1 || n > 2147483647LL || d < 1 || d > 65536)
    return fail(nullptr, KKM_ERR_ARG, "bad sizes n=%lld d=%d", (long long)n, d);
  if (kind != KKM_LINEAR && kind != KKM_POLY && kind != KKM_GAUSS)
    return fail(nullptr, KKM_ERR_ARG, "bad kind=%d", kind);
  if (requested_mode < KKM_MODE_AUTO || requested_mode > KKM_MODE_PACKED)
    return fail(nullptr, KKM_ERR_ARG, "bad mode=%d", requested_mode);
  if (requested_mode == KKM_MODE_PACKED && k_known && k > KKM_PACKED_MAX_K)
    return fail(nullptr, KKM_ERR_ARG, "packed storage handles k <= %d, not %d", KKM_PACKED_MAX_K, k);
  if (storage != KKM_STORE_F32 && storage != KKM_STORE_F16) return fail(nullptr, KKM_ERR_ARG, "bad storage=%d", storage);
  auto need_for = [&](int m) {
    const Sizes s = sizes_for(n, d, m);
    const size_t scales = row_scaled(m, storage, kind) ? (size_t)n * 4 + 256 : 0;
    return staged_bytes(s) + ws_bytes(s, k, m) + 4096 + k_bytes(s, m, storage) + scales;
  };
  auto fits = [&](int m) { return need_for(m) <= mem_budget; };
  int mode = requested_mode;
  if (mode == KKM_MODE_AUTO) {
    if (k_known && k <= KKM_PACKED_FAST_K && fits(KKM_MODE_PACKED)) mode = KKM_MODE_PACKED;
    else if (fits(KKM_MODE_RESIDENT)) mode = KKM_MODE_RESIDENT;
    else if (!k_known && fits(KKM_MODE_PACKED)) mode = KKM_MODE_PACKED;
    else mode = KKM_MODE_ONTHEFLY;
  }
  const size_t need = need_for(mode);
  if (mode_out) *mode_out = mode;
  if (bytes_out) *bytes_out = need;
  static const char* names[] = {"auto", "resident", "on-the-fly", "packed"};
  if (need > mem_budget)
    return fail(nullptr, KKM_ERR_OOM, "%s mode needs %zu bytes, budget %zu", names[mode], need, mem_budget);
  return KKM_OK;
}

}  // namespace

extern "C" {

int kkm_abi_version(void) { return KKM_ABI_VERSION; }

const char* kkm_last_error(const kkm_ctx* ctx) { return ctx ? ctx->err.c_str() : g_noctx_err.c_str(); }

const char* kkm_last_warning(const kkm_ctx* ctx) { return ctx ? ctx->warn.c_str() : g_noctx_warn.c_str(); }

int kkm_check_build_args(int64_t n, int32_t d, int32_t kind, const kkm_params* p) {
  if (n < 1 || n > 2147483647LL) return fail(nullptr, KKM_ERR_ARG, "n=%lld must be in [1, 2^31-1]", (long long)n);
  if (d < 1 || d > 65536) return fail(nullptr, KKM_ERR_ARG, "d=%d must be in [1, 65536]", d);
  if (kind != KKM_LINEAR && kind != KKM_POLY && kind != KKM_GAUSS)
    return fail(nullptr, KKM_ERR_ARG, "kind=%d is not LINEAR(0), POLY(1) or GAUSS(2)", kind);
  if (!p) return fail(nullptr, KKM_ERR_ARG, "params is NULL");
  if (p->mode < KKM_MODE_AUTO || p->mode > KKM_MODE_PACKED)
    return fail(nullptr, KKM_ERR_ARG, "mode=%d is not AUTO(0), RESIDENT(1), ONTHEFLY(2) or PACKED(3)", p->mode);
  if (p->storage != KKM_STORE_F32 && p->storage != KKM_STORE_F16)
    return fail(nullptr, KKM_ERR_ARG, "storage=%d is not F32(0) or F16(1)", p->storage);
  if (p->k_hint < 0 || p->k_hint > KKM_MAX_K)
    return fail(nullptr, KKM_ERR_ARG, "k_hint=%d must be 0 (unknown) or in [1, %d]", p->k_hint, KKM_MAX_K);
  g_noctx_warn.clear();
  if (kind == KKM_POLY) {
    if (!(std::isfinite(p->gamma) && std::isfinite(p->coef0)))
      return fail(nullptr, KKM_ERR_ARG, "polynomial gamma and coef0 must be finite");
    if (p->degree < 1 || p->degree > 16)
      return fail(nullptr, KKM_ERR_ARG, "polynomial degree=%d must be in [1, 16]", p->degree);
    // (gamma x.y + c)^p is a positive semidefinite kernel for gamma >= 0,
    // c >= 0 and integer p (a sum of products of PSD kernels); otherwise K
    // may have negative eigenvalues and J need not fall from update to update.
    if (p->coef0 < 0.f || p->gamma < 0.f) {
      char buf[256];
      snprintf(buf, sizeof buf,
               "polynomial kernel with gamma=%g, coef0=%g is not positive semidefinite: the objective J "
               "need not decrease from update to update",
               (double)p->gamma, (double)p->coef0);
      g_noctx_warn = buf;
    }
  }
  if (kind == KKM_GAUSS && !(p->gamma > 0.f && std::isfinite(p->gamma)))
    return fail(nullptr, KKM_ERR_ARG, "Gaussian gamma=%g must be finite and > 0", (double)p->gamma);
  return KKM_OK;
}

int kkm_check_iterate_args(int64_t n, int32_t k, int32_t max_iter) {
  if (k < 1 || k > KKM_MAX_K) return fail(nullptr, KKM_ERR_ARG, "k=%d must be in [1, %d]", k, KKM_MAX_K);
  if ((int64_t)k > n) return fail(nullptr, KKM_ERR_ARG, "k=%d exceeds n=%lld", k, (long long)n);
  if (max_iter < 0) return fail(nullptr, KKM_ERR_ARG, "max_iter=%d must be >= 0", max_iter);
  return KKM_OK;
}

int kkm_plan(int64_t n, int32_t d, int32_t k, int32_t kind, size_t mem_budget, int32_t requested_mode,
             int32_t storage, int32_t* mode_out, size_t* bytes_out) {
  if (n < 1 || n > 2147483647LL || d < 1 || d > 65536)
    return fail(nullptr, KKM_ERR_ARG, "bad sizes n=%lld d=%d", (long long)n, d);
  if (k < 1 || k > KKM_MAX_K || (int64_t)k > n) return fail(nullptr, KKM_ERR_ARG, "bad k=%d", k);
  return plan_impl(n, d, k, true, kind, mem_budget, requested_mode, storage, mode_out, bytes_out);
}

int kkm_create(kkm_ctx** out, void* hip_stream, size_t mem_budget) {
  if (!out) return fail(nullptr, KKM_ERR_ARG, "out is NULL");
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(nullptr, KKM_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (mem_budget == 0) {
    size_t freeb = 0, totalb = 0;
    e = hipMemGetInfo(&freeb, &totalb);
    if (e != hipSuccess) return fail(nullptr, KKM_ERR_HIP, "hipMemGetInfo: %s", hipGetErrorString(e));
    mem_budget = (size_t)((double)freeb * 0.95);
  }
  void* scr = nullptr;
  e = scratch_address(dev, &scr);
  if (e != hipSuccess) return fail(nullptr, KKM_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
  kkm_ctx* c = new kkm_ctx();
  c->stream = (hipStream_t)hip_stream;
  c->device = dev;
  c->scratch = scr;
  c->budget = mem_budget;
  *out = c;
  return KKM_OK;
}

int kkm_destroy(kkm_ctx* c) {
  if (!c) return KKM_OK;
  (void)hipStreamSynchronize(c->stream);
  collect_timing(c);
  free_build(c);
  for (hipEvent_t e : c->pool) (void)hipEventDestroy(e);
  delete c;
  return KKM_OK;
}

}  // extern "C"

namespace {

// The build of the full K (pc1 = 0) or of the block K[pr0 : pr1, pc0 : pc1)
// of one GPU's share (resident, fp32).
int build_impl(kkm_ctx* c, const float* X, int64_t n, int32_t d, int32_t kind, const kkm_params* params,
               int64_t pr0, int64_t pr1, int64_t pc0, int64_t pc1) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  c->warn.clear();
  if (kkm_check_build_args(n, d, kind, params) != KKM_OK) return fail(c, KKM_ERR_ARG, "%s", g_noctx_err.c_str());
  c->warn = g_noctx_warn;
  if (!X) return fail(c, KKM_ERR_ARG, "X is NULL");
  const bool panel = pc1 > 0;
  int32_t mode = KKM_MODE_RESIDENT;
  size_t need = 0;
  if (panel) {
    if (params->storage != KKM_STORE_F32) return fail(c, KKM_ERR_ARG, "a block of K is stored in fp32");
  } else {
    // plan with the caller's k hint (else k = 1 sizes the scratch and the
    // mode is picked without k): the k-dependent scratch is sized when
    // kkm_iterate is called
    size_t held_by_build = 0;
    for (const Alloc& a : c->build_allocs) held_by_build += a.bytes;
    for (const Alloc& a : c->ws_allocs) held_by_build += a.bytes;
    for (const Alloc& a : c->hist_allocs) held_by_build += a.bytes;
    const size_t budget_left = c->budget - std::min(c->budget, c->held - std::min(c->held, held_by_build));
    const int32_t kh = std::min<int64_t>(params->k_hint, n);
    if (plan_impl(n, d, kh > 0 ? kh : 1, kh > 0, kind, budget_left, params->mode, params->storage, &mode,
                  &need) != KKM_OK)
      return fail(c, KKM_ERR_OOM, "%s", g_noctx_err.c_str());
  }
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  collect_timing(c);
  // A rebuild of the same shape keeps every buffer (K alone can be 160 GB,
  // and allocating it costs far more than building it).
  const int storage = (mode == KKM_MODE_RESIDENT || mode == KKM_MODE_PACKED) ? params->storage : KKM_STORE_F32;
  // (a block of the same shape elsewhere in K also keeps them)
  const bool reuse = c->built && c->sz.n == n && c->d == d && c->mode == mode && c->kind == kind &&
                     c->storage == storage && (c->pc1 > 0) == panel && c->pr1 - c->pr0 == pr1 - pr0 &&
                     c->pc1 - c->pc0 == pc1 - pc0;
  if (!reuse) free_build(c);

  c->sz = sizes_for(n, d, mode);
  if (panel) {  // the block's columns: a multiple of kTile, so its tiles store whole
    c->sz.ld = round_up(pc1 - pc0, kTile);
    c->sz.nstripes = (int)((c->sz.ld + kStripe - 1) / kStripe);
  }
  c->wsz = c->sz;
  if (panel) {  // K and the scratch hold the block's rows
    c->wsz.n = pr1 - pr0;
    c->wsz.n_pad = round_up(pr1 - pr0, kTile);
    c->wsz.nblk = (pr1 - pr0 + kBlk - 1) / kBlk;
  }
  c->pr0 = pr0;
  c->pr1 = pr1;
  c->pc0 = pc0;
  c->pc1 = pc1;
  c->panel_e = false;
  c->d = d;
  c->kind = kind;
  c->mode = mode;
  c->storage = storage;
  c->params = *params;
  KappaParams& kp = c->kp;
  kp.kind = kind;
  kp.gamma = params->gamma;
  kp.coef0 = params->coef0;
  kp.degree = params->degree;
  kp.neg_g_log2e = (float)(-(double)params->gamma * 1.4426950408889634);
  kp.fix_scale = (float)((double)params->gamma * kFixAcc * std::ldexp(1.0, -24));
  kp.fix_tol = kFixTol;
  kp.m2c = -2.0f * kp.neg_g_log2e;
  kp.fix_uthr = (float)((double)kp.neg_g_log2e * kFixTol / (double)kp.fix_scale);

  const Sizes& s = c->sz;
  int rc;
  void* p = nullptr;
  if (!reuse) {
    if ((rc = dalloc(c, &p, staged_bytes(s), c->build_allocs, "staged points"))) return rc;
    c->Xp = (float*)p;
    c->nrm = c->Xp + (size_t)s.n_pad * s.d_pad;
    c->diagK = c->nrm + s.n_pad;
    c->bmax = c->diagK + s.n;
    if ((rc = dalloc(c, &p, 64, c->build_allocs, "trace"))) return rc;
    c->trK = (double*)p;
    c->maxnrm = (unsigned*)((char*)p + 8);
    const bool stores_k = mode == KKM_MODE_RESIDENT || mode == KKM_MODE_PACKED;
    if (stores_k) {
      const size_t kb = k_bytes(c->wsz, mode, storage);
      if ((rc = dalloc(c, &p, kb, c->build_allocs, "kernel matrix K", kb >= kContiguousFromK))) return rc;
      c->K = p;
    }
    if (row_scaled(mode, storage, kind)) {
      if ((rc = dalloc(c, &p, (size_t)n * 4, c->build_allocs, "row scales"))) return rc;
      c->kw = (float*)p;
    }
  }
  // The Gaussian fix-up list takes up to a quarter of the room the budget
  // leaves.  It is needed only while building: the first iteration scratch
  // that does not fit beside it releases it (release_fix_list), and a
  // rebuild then makes it again here.
  if (kind == KKM_GAUSS && (mode == KKM_MODE_RESIDENT || mode == KKM_MODE_PACKED) && !c->fix_list) {
    const long long upper = panel ? (long long)((pr1 - pr0) * (pc1 - pc0)) : (long long)(n * (n - 1) / 2);
    long long cap = std::min<long long>(upper, std::max<long long>(1LL << 20, 512LL * n));
    const size_t room = c->budget > c->held ? c->budget - c->held : 0;
    cap = std::min<long long>(cap, (long long)(room / 4 / sizeof(int2)));
    cap = std::max<long long>(cap / kFixSegs, 1) * kFixSegs;
    if ((rc = dalloc(c, &p, (size_t)cap * sizeof(int2) + kFixSegs * 8, c->build_allocs, "fix-up list")))
      return rc;
    c->fix_list = (int2*)p;
    c->fix_count = (unsigned long long*)((char*)p + (size_t)cap * sizeof(int2));
    c->fix_cap = cap;
  }
  if ((rc = run(c, KKM_PHASE_STAGE, "zero", [&] { return launch_zero_ints((int*)c->maxnrm, 1, c->stream); })))
    return rc;
  if ((rc = run(c, KKM_PHASE_STAGE, "stage", [&] {
         return launch_stage(X, n, d, s.d_pad, s.n_pad, c->Xp, c->nrm, c->maxnrm, c->stream);
       })))
    return rc;
  c->fixups = -1;  // read from the device on demand
  if (c->fix_count && (rc = run(c, KKM_PHASE_FIXUP, "zero", [&] {
        return launch_zero_ints((int*)c->fix_count, 2 * kFixSegs, c->stream);
      })))
    return rc;
  c->built = true;  // buffers exist from here on; free_build releases them

  if (mode == KKM_MODE_ONTHEFLY) {
    if ((rc = run(c, KKM_PHASE_STAGE, "diag", [&] { return launch_diag_from_norms(c->nrm, n, kp, c->diagK, c->stream); })))
      return rc;
    return run(c, KKM_PHASE_OTHER, "trace", [&] { return launch_trace(c->diagK, n, c->trK, c->stream); });
  }
  const bool f16 = storage == KKM_STORE_F16;
  if (c->kw && (rc = run(c, KKM_PHASE_STAGE, "row_scales", [&] {
        return launch_row_scales(c->nrm, c->maxnrm, n, kp, c->kw, c->stream);
      })))
    return rc;
  if (!panel && kind == KKM_GAUSS &&
      (rc = run(c, KKM_PHASE_STAGE, "blockmax", [&] { return launch_blockmax(c->nrm, s.n_pad / kTile, c->bmax, c->stream); })))
    return rc;
  if ((rc = run(c, KKM_PHASE_GEMM, "gemm_kappa", [&] {
         if (panel)
           return launch_gemm_kappa_panel(c->Xp, c->nrm, c->maxnrm, n, s.d_pad, pr0, pr1, pc0, pc1, s.ld, kp,
                                          (float*)c->K, c->diagK, c->fix_list, c->fix_count,
                                          c->fix_cap / kFixSegs, c->stream);
         // the build divides by the row bounds only for binary16 storage
         return launch_gemm_kappa(c->Xp, c->nrm, c->maxnrm, n, s.d_pad, s.ld, mode == KKM_MODE_PACKED, f16,
                                  f16 ? c->kw : nullptr, kp, c->K, c->diagK, c->fix_list, c->fix_count,
                                  c->fix_cap / kFixSegs, c->bmax, c->stream);
       })))
    return rc;
  if (kind == KKM_GAUSS &&
      (rc = run(c, KKM_PHASE_FIXUP, "gauss_fixup", [&] {
         return launch_gauss_fixup(c->Xp, c->nrm, n, s.d_pad, s.ld, mode == KKM_MODE_PACKED, f16, kp,
                                   c->fix_list, c->fix_count, c->fix_cap / kFixSegs, c->K, c->stream, pr0, pr1,
                                   pc0, pc1);
       })))
    return rc;
  // A panel's tiles set diag K for its points.  Another block's diagonal may
  // lie elsewhere, so diag K of every point comes from the norms, as the
  // on-the-fly mode takes it; no trace.
  if (panel && (pr0 > 0 || pr1 < n))
    return run(c, KKM_PHASE_STAGE, "diag", [&] { return launch_diag_from_norms(c->nrm, n, kp, c->diagK, c->stream); });
  if (panel) return KKM_OK;
  return run(c, KKM_PHASE_OTHER, "trace", [&] { return launch_trace(c->diagK, n, c->trK, c->stream); });
}

}  // namespace

extern "C" {

int kkm_build_kernel(kkm_ctx* c, const float* X, int64_t n, int32_t d, int32_t kind, const kkm_params* params) {
  return build_impl(c, X, n, d, kind, params, 0, 0, 0, 0);
}

int kkm_build_panel(kkm_ctx* c, const float* X, int64_t n, int32_t d, int32_t kind, const kkm_params* params,
                    int64_t c0, int64_t c1) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (c0 < 0 || c0 % kTile || c1 <= c0 || c1 > n)
    return fail(c, KKM_ERR_ARG, "bad panel [%lld, %lld): needs 0 <= c0 < c1 <= n=%lld, c0 a multiple of %d",
                (long long)c0, (long long)c1, (long long)n, kTile);
  if (round_up(c1 - c0, kTile) >= kMaxKStride)
    return fail(c, KKM_ERR_ARG, "panel of %lld columns: at most %lld fit the K build's 32-bit store offsets",
                (long long)(c1 - c0), (long long)(kMaxKStride - kTile));
  return build_impl(c, X, n, d, kind, params, 0, n, c0, c1);
}

int kkm_build_block(kkm_ctx* c, const float* X, int64_t n, int32_t d, int32_t kind, const kkm_params* params,
                    int64_t r0, int64_t r1, int64_t c0, int64_t c1) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (r0 < 0 || r0 % kTile || r1 <= r0 || r1 > n || c0 < 0 || c0 % kTile || c1 <= c0 || c1 > n)
    return fail(c, KKM_ERR_ARG,
                "bad block [%lld, %lld) x [%lld, %lld): needs 0 <= start < end <= n=%lld on both sides, "
                "starts multiples of %d",
                (long long)r0, (long long)r1, (long long)c0, (long long)c1, (long long)n, kTile);
  if (round_up(c1 - c0, kTile) >= kMaxKStride)
    return fail(c, KKM_ERR_ARG, "block of %lld columns: at most %lld fit the K build's 32-bit store offsets",
                (long long)(c1 - c0), (long long)(kMaxKStride - kTile));
  return build_impl(c, X, n, d, kind, params, r0, r1, c0, c1);
}

int kkm_panel_spmm(kkm_ctx* c, const int32_t* cl, int32_t k, double* zpart, int32_t* counts) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!c->built || c->pc1 == 0 || c->pr0 != 0 || c->pr1 != c->sz.n)
    return fail(c, KKM_ERR_STATE, "no panel (all rows of K) built on this context");
  if (kkm_check_iterate_args(c->sz.n, k, 1) != KKM_OK) return fail(c, KKM_ERR_ARG, "%s", g_noctx_err.c_str());
  if (!cl || !zpart) return fail(c, KKM_ERR_ARG, "cl or zpart is NULL");
  int rc;
  c->panel_e = false;
  if ((rc = ensure_ws(c, k, 1))) return rc;
  if ((rc = label_pass(c, cl))) return rc;  // sizes of cl in counts[0], per-block histograms
  IterBufs& b = c->ib;
  if ((rc = run(c, KKM_PHASE_SCATTER, "scatter", [&] {
         return launch_scatter(b, cl, c->counts[0], c->counts[1], c->changed, c->stream);
       })))
    return rc;
  if ((rc = run(c, KKM_PHASE_SPMM, "spmm_onehot", [&] { return launch_spmm_onehot(c->K, b, c->stream); })))
    return rc;
  if ((rc = run(c, KKM_PHASE_REDUCE, "spmm_reduce", [&] { return launch_spmm_reduce(b, cl, c->stream); })))
    return rc;
  std::vector<double> parts((size_t)k * b.nzpart);
  int status = 0;
  HIP_TRY(c, hipMemcpyAsync(parts.data(), b.zpart, parts.size() * sizeof(double), hipMemcpyDeviceToHost, c->stream),
          "read z parts");
  if (counts)
    HIP_TRY(c, hipMemcpyAsync(counts, c->counts[0], (size_t)k * 4, hipMemcpyDeviceToHost, c->stream), "read sizes");
  HIP_TRY(c, hipMemcpyAsync(&status, b.status, sizeof status, hipMemcpyDeviceToHost, c->stream), "read status");
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  if ((rc = status_error(c, status))) return rc;
  for (int j = 0; j < k; ++j) {  // the stripes in order
    double zs = 0.0;
    for (int x = 0; x < b.nzpart; ++x) zs += parts[(size_t)j * b.nzpart + x];
    zpart[j] = zs;
  }
  c->panel_e = true;
  return KKM_OK;
}

int kkm_panel_assign(kkm_ctx* c, int32_t k, const double* z, int32_t* cl_out, float* E_out, int32_t* counts_out) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!c->built || c->pc1 == 0 || c->pr0 != 0 || c->pr1 != c->sz.n)
    return fail(c, KKM_ERR_STATE, "no panel (all rows of K) built on this context");
  if (!c->panel_e || c->ib.k != k) return fail(c, KKM_ERR_STATE, "kkm_panel_spmm with this k must come first");
  if (!z || !cl_out) return fail(c, KKM_ERR_ARG, "z or cl_out is NULL");
  IterBufs& b = c->ib;
  // z goes to the device through the (now read) reduction parts: k floats
  std::vector<float> zf((size_t)k);
  for (int j = 0; j < k; ++j) zf[j] = (float)z[j];
  float* zd = (float*)b.zpart;
  int rc;
  HIP_TRY(c, hipMemcpyAsync(zd, zf.data(), (size_t)k * 4, hipMemcpyHostToDevice, c->stream), "write z");
  if ((rc = run(c, KKM_PHASE_ASSIGN, "zero", [&] { return launch_zero_ints(c->counts[1], k, c->stream); })))
    return rc;
  if ((rc = run(c, KKM_PHASE_ASSIGN, "panel_assign", [&] {
         return launch_panel_assign(b, zd, c->counts[0], cl_out, c->counts[1], E_out, c->stream);
       })))
    return rc;
  if (counts_out)
    HIP_TRY(c, hipMemcpyAsync(counts_out, c->counts[1], (size_t)k * 4, hipMemcpyDeviceToHost, c->stream),
            "read sizes");
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  return KKM_OK;
}

int kkm_block_spmm(kkm_ctx* c, const int32_t* cl, int32_t k, float* E_out) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!c->built || c->pc1 == 0) return fail(c, KKM_ERR_STATE, "no block of K built on this context");
  if (kkm_check_iterate_args(c->sz.n, k, 1) != KKM_OK) return fail(c, KKM_ERR_ARG, "%s", g_noctx_err.c_str());
  if (!cl || !E_out) return fail(c, KKM_ERR_ARG, "cl or E_out is NULL");
  int rc;
  c->panel_e = false;
  if ((rc = ensure_ws(c, k, 1))) return rc;
  if ((rc = label_pass(c, cl))) return rc;  // the block's rows: sizes in counts[0], per-block histograms
  IterBufs& b = c->ib;
  if ((rc = run(c, KKM_PHASE_SCATTER, "scatter", [&] {
         return launch_scatter(b, cl, c->counts[0], c->counts[1], c->changed, c->stream);
       })))
    return rc;
  if ((rc = run(c, KKM_PHASE_SPMM, "spmm_onehot", [&] { return launch_spmm_onehot(c->K, b, c->stream); })))
    return rc;
  if ((rc = run(c, KKM_PHASE_REDUCE, "block_out", [&] { return launch_block_out(b, E_out, c->stream); })))
    return rc;
  int status = 0;
  HIP_TRY(c, hipMemcpyAsync(&status, b.status, sizeof status, hipMemcpyDeviceToHost, c->stream), "read status");
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  return status_error(c, status);
}

namespace {
// A piece [a0, a1) of the block's columns, for the calls that follow the
// caller's reduce-scatter.
int check_piece(kkm_ctx* c, int64_t a0, int64_t a1, int32_t k) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!c->built || c->pc1 == 0) return fail(c, KKM_ERR_STATE, "no block of K built on this context");
  if (kkm_check_iterate_args(c->sz.n, k, 1) != KKM_OK) return fail(c, KKM_ERR_ARG, "%s", g_noctx_err.c_str());
  if (a0 < c->pc0 || a1 <= a0 || a1 > c->pc1)
    return fail(c, KKM_ERR_ARG, "bad piece [%lld, %lld): needs %lld <= a0 < a1 <= %lld, the block's columns",
                (long long)a0, (long long)a1, (long long)c->pc0, (long long)c->pc1);
  return KKM_OK;
}
}  // namespace

int kkm_block_zpart(kkm_ctx* c, const float* E, const int32_t* cl, int64_t a0, int64_t a1, int32_t k,
                    double* zpart, int32_t* counts) {
  int rc;
  if ((rc = check_piece(c, a0, a1, k))) return rc;
  if (!E || !cl || !zpart || !counts) return fail(c, KKM_ERR_ARG, "E, cl, zpart or counts is NULL");
  if ((rc = ensure_ws(c, k, 1))) return rc;
  IterBufs& b = c->ib;
  const int64_t m = a1 - a0;
  const int ng = (int)((m + 1023) / 1024);  // workgroups: at most one per column stripe, so <= nzpart
  if ((rc = run(c, KKM_PHASE_LABELS, "zero", [&] { return launch_zero_ints(c->counts[0], k, c->stream); })))
    return rc;
  if ((rc = run(c, KKM_PHASE_LABELS, "zero", [&] { return launch_zero_ints(b.status, 1, c->stream); })))
    return rc;
  if ((rc = run(c, KKM_PHASE_REDUCE, "cols_zpart", [&] {
         return launch_cols_zpart(E, cl, m, k, b.zpart, b.nzpart, c->counts[0], b.status, c->stream);
       })))
    return rc;
  std::vector<double> parts((size_t)k * b.nzpart);
  int status = 0;
  HIP_TRY(c, hipMemcpyAsync(parts.data(), b.zpart, parts.size() * sizeof(double), hipMemcpyDeviceToHost, c->stream),
          "read z parts");
  HIP_TRY(c, hipMemcpyAsync(counts, c->counts[0], (size_t)k * 4, hipMemcpyDeviceToHost, c->stream), "read sizes");
  HIP_TRY(c, hipMemcpyAsync(&status, b.status, sizeof status, hipMemcpyDeviceToHost, c->stream), "read status");
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  if ((rc = status_error(c, status))) return rc;
  for (int j = 0; j < k; ++j) {  // the workgroups in order
    double zs = 0.0;
    for (int g = 0; g < ng; ++g) zs += parts[(size_t)j * b.nzpart + g];
    zpart[j] = zs;
  }
  return KKM_OK;
}

int kkm_block_assign(kkm_ctx* c, const float* E, int64_t a0, int64_t a1, int32_t k, const double* z,
                     const int32_t* counts, int32_t* cl_out, int32_t* counts_out) {
  int rc;
  if ((rc = check_piece(c, a0, a1, k))) return rc;
  if (!E || !z || !counts || !cl_out) return fail(c, KKM_ERR_ARG, "E, z, counts or cl_out is NULL");
  for (int j = 0; j < k; ++j)
    if (counts[j] < 0) return fail(c, KKM_ERR_ARG, "counts[%d] = %d is negative", j, counts[j]);
  if ((rc = ensure_ws(c, k, 1))) return rc;
  IterBufs& b = c->ib;
  c->panel_e = false;  // z and the sizes below take the panel's places
  std::vector<float> zf((size_t)k);
  for (int j = 0; j < k; ++j) zf[j] = (float)z[j];
  float* zd = (float*)b.zpart;
  HIP_TRY(c, hipMemcpyAsync(zd, zf.data(), (size_t)k * 4, hipMemcpyHostToDevice, c->stream), "write z");
  HIP_TRY(c, hipMemcpyAsync(c->counts[0], counts, (size_t)k * 4, hipMemcpyHostToDevice, c->stream), "write sizes");
  if ((rc = run(c, KKM_PHASE_ASSIGN, "zero", [&] { return launch_zero_ints(c->counts[1], k, c->stream); })))
    return rc;
  if ((rc = run(c, KKM_PHASE_ASSIGN, "cols_assign", [&] {
         return launch_cols_assign(E, k, 1, c->diagK + a0, a1 - a0, k, zd, c->counts[0], cl_out, c->counts[1],
                                   nullptr, c->stream);
       })))
    return rc;
  if (counts_out)
    HIP_TRY(c, hipMemcpyAsync(counts_out, c->counts[1], (size_t)k * 4, hipMemcpyDeviceToHost, c->stream),
            "read sizes");
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  return KKM_OK;
}

}  // extern "C"

namespace {

// The loop of kkm_iterate on per-update scratch already laid out (c->ib and
// the id, size and history buffers).
int iterate_loop(kkm_ctx* c, int32_t* V, int32_t k, int32_t max_iter, double tol, int32_t* iters_done,
                 double* obj_hist) {
  int rc;
  if ((rc = label_pass(c, V))) return rc;
  const int* cur = V;
  int t = 0, status = 0;
  double Jprev = 0.0;
  for (; t < max_iter; ++t) {
    int* nxt = c->clbuf[t & 1];
    if ((rc = one_update(c, t, cur, nxt, nullptr, nullptr))) return rc;
    cur = nxt;
    if (tol >= 0.0) {
      int chg = 0;
      double J = 0.0;
      HIP_TRY(c, hipMemcpyAsync(&chg, c->changed + t, sizeof chg, hipMemcpyDeviceToHost, c->stream), "read changes");
      HIP_TRY(c, hipMemcpyAsync(&J, c->obj + t, sizeof J, hipMemcpyDeviceToHost, c->stream), "read objective");
      HIP_TRY(c, hipMemcpyAsync(&status, c->ib.status, sizeof status, hipMemcpyDeviceToHost, c->stream), "read status");
      HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
      if ((rc = status_error(c, status))) return rc;
      bool stop = chg == 0;
      if (!stop && tol > 0.0 && t > 0 && (Jprev - J) <= tol * std::fabs(Jprev)) stop = true;
      Jprev = J;
      if (stop) {
        ++t;
        break;
      }
    }
  }
  if (t > 0)
    HIP_TRY(c, hipMemcpyAsync(V, cur, (size_t)c->sz.n * 4, hipMemcpyDeviceToDevice, c->stream), "copy ids");
  if (obj_hist && t > 0)
    HIP_TRY(c, hipMemcpyAsync(obj_hist, c->obj, (size_t)t * sizeof(double), hipMemcpyDeviceToHost, c->stream),
            "read objective history");
  HIP_TRY(c, hipMemcpyAsync(&status, c->ib.status, sizeof status, hipMemcpyDeviceToHost, c->stream), "read status");
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  if ((rc = status_error(c, status))) return rc;
  if (iters_done) *iters_done = t;
  return KKM_OK;
}

}  // namespace

extern "C" {

int kkm_iterate(kkm_ctx* c, int32_t* V, int32_t k, int32_t max_iter, double tol, int32_t* iters_done,
                double* obj_hist) {
  int rc;
  if ((rc = check_ready(c, k, max_iter))) return rc;
  if (!V) return fail(c, KKM_ERR_ARG, "V is NULL");
  if (iters_done) *iters_done = 0;
  if ((rc = ensure_ws(c, k, max_iter))) return rc;
  return iterate_loop(c, V, k, max_iter, tol, iters_done, obj_hist);
}

int kkm_iterate_noalloc(kkm_ctx* c, int32_t* V, int32_t k, int32_t max_iter, double tol, int32_t* iters_done,
                        double* obj_hist) {
  int rc;
  if ((rc = check_ready(c, k, max_iter))) return rc;
  if (!V) return fail(c, KKM_ERR_ARG, "V is NULL");
  if (iters_done) *iters_done = 0;
  if (!c->scratch) return fail(c, KKM_ERR_STATE, "the static scratch of this device is not mapped");
  const size_t ws = round_up((int64_t)ws_bytes(c->wsz, k, c->mode), 256);
  const int cap = std::max(max_iter, 1);
  const size_t hist = (size_t)cap * 12 + 512;
  if (ws + hist > KKM_NOALLOC_SCRATCH_BYTES)
    return fail(c, KKM_ERR_ARG,
                "this problem (n=%lld, k=%d, %s storage, %d updates) needs %zu bytes of scratch; the static "
                "scratch holds %zu: use kkm_iterate",
                (long long)c->wsz.n, k, c->mode == KKM_MODE_PACKED ? "packed" : c->mode == KKM_MODE_RESIDENT ? "full" : "no",
                max_iter, ws + hist, (size_t)KKM_NOALLOC_SCRATCH_BYTES);
  // The context's own scratch (if any) is set aside for this call and put
  // back after it; no launch is bracketed by events (creating one may allocate).
  const SavedWs saved = save_ws(c);
  const int32_t timing = c->timing;
  c->timing = 0;
  rc = carve_from(c, k, c->scratch);
  if (!rc) {
    c->obj = (double*)((char*)c->scratch + ws);
    c->changed = (int*)((char*)c->obj + (size_t)cap * 8);
    c->iter_ws = cap;
    rc = iterate_loop(c, V, k, max_iter, tol, iters_done, obj_hist);
  }
  c->timing = timing;
  restore_ws(c, saved);
  return rc;
}

int kkm_step(kkm_ctx* c, const int32_t* cl_in, int32_t k, float* E, float* z, float* D, int32_t* cl_out,
             int32_t* counts_out, double* J) {
  int rc;
  if ((rc = check_ready(c, k, 1))) return rc;
  if (!cl_in) return fail(c, KKM_ERR_ARG, "cl_in is NULL");
  if ((rc = ensure_ws(c, k, 1))) return rc;
  if ((rc = label_pass(c, cl_in))) return rc;
  int* nxt = cl_out ? cl_out : c->clbuf[0];
  if ((rc = one_update(c, 0, cl_in, nxt, z, D))) return rc;
  if (E && (rc = run(c, KKM_PHASE_OTHER, "et_to_e", [&] { return launch_et_to_e(c->ib, c->counts[0], c->epos, E, c->stream); })))
    return rc;
  if (counts_out)
    HIP_TRY(c, hipMemcpyAsync(counts_out, c->counts[0], (size_t)k * 4, hipMemcpyDeviceToDevice, c->stream), "copy counts");
  double Jv = 0.0;
  int status = 0;
  HIP_TRY(c, hipMemcpyAsync(&Jv, c->obj, sizeof(double), hipMemcpyDeviceToHost, c->stream), "read objective");
  HIP_TRY(c, hipMemcpyAsync(&status, c->ib.status, sizeof status, hipMemcpyDeviceToHost, c->stream), "read status");
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  if ((rc = status_error(c, status))) return rc;
  if (J) *J = Jv;
  return KKM_OK;
}

int kkm_objective(kkm_ctx* c, const int32_t* V, int32_t k, double* J) {
  if (!J) return fail(c, KKM_ERR_ARG, "J is NULL");
  return kkm_step(c, V, k, nullptr, nullptr, nullptr, nullptr, nullptr, J);
}

int kkm_init_kmeanspp(kkm_ctx* c, int32_t k, const double* u, int32_t* centers_out, int32_t* V) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!c->built) return fail(c, KKM_ERR_STATE, "no kernel matrix built on this context");
  const int64_t n = c->sz.n;
  if (k < 1 || k > KKM_MAX_K || (int64_t)k > n)
    return fail(c, KKM_ERR_ARG, "k=%d must be in [1, min(n=%lld, %d)]", k, (long long)n, KKM_MAX_K);
  if (!u) return fail(c, KKM_ERR_ARG, "u is NULL");
  if (!V) return fail(c, KKM_ERR_ARG, "V is NULL");
  for (int t = 0; t < k; ++t)
    if (!(u[t] >= 0.0 && u[t] < 1.0)) return fail(c, KKM_ERR_ARG, "u[%d]=%g is outside [0, 1)", t, u[t]);
  if (!c->sd_kd) {
    const size_t nb = (size_t)seed_blocks(n);
    const size_t bytes = 4 * (((size_t)n * 4 + 255) / 256 * 256) + (nb * 8 + 255) / 256 * 256 + KKM_MAX_K * 4;
    void* base = nullptr;
    int rc = dalloc(c, &base, bytes, c->seed_allocs, "seeding scratch");
    if (rc) return rc;
    char* p = (char*)base;
    auto take = [&](size_t b) {
      char* r = p;
      p += (b + 255) / 256 * 256;
      return (void*)r;
    };
    c->sd_kd = (float*)take((size_t)n * 4);
    c->sd_D = (float*)take((size_t)n * 4);
    c->sd_best = (float*)take((size_t)n * 4);
    c->sd_bestc = (int*)take((size_t)n * 4);
    c->sd_bsum = (double*)take(nb * 8);
    c->sd_centers = (int*)take((size_t)KKM_MAX_K * 4);
  }
  const int c_first = (int)std::min<int64_t>((int64_t)std::floor(u[0] * (double)n), n - 1);
  for (int t = 0; t < k; ++t) {
    if (t > 0) {
      int rc = run(c, KKM_PHASE_SEED, "kpp_select", [&] {
        return launch_kpp_select(c->sd_D, c->sd_bsum, n, u[t], c->sd_centers, t, c->stream);
      });
      if (rc) return rc;
    }
    int rc = run(c, KKM_PHASE_SEED, "kpp_dist", [&] {
      return launch_kpp_dist(c->Xp, n, c->sz.d_pad, c->kp, c->sd_centers, t, c_first, c->sd_kd, c->sd_D,
                             c->sd_best, c->sd_bestc, c->sd_bsum, t == k - 1 ? V : nullptr, c->stream);
    });
    if (rc) return rc;
  }
  if (centers_out)
    HIP_TRY(c, hipMemcpyAsync(centers_out, c->sd_centers, (size_t)k * 4, hipMemcpyDeviceToHost, c->stream),
            "copy centers");
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  return KKM_OK;
}

int kkm_copy_kernel_rows(kkm_ctx* c, int64_t r0, int64_t r1, float* out) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!c->built) return fail(c, KKM_ERR_STATE, "no kernel matrix built on this context");
  const int64_t lo = c->pc1 > 0 ? c->pr0 : 0, hi = c->pc1 > 0 ? c->pr1 : c->sz.n;
  if (!out || r0 < lo || r1 > hi || r0 > r1)
    return fail(c, KKM_ERR_ARG, "bad row range [%lld, %lld): the stored rows are [%lld, %lld)", (long long)r0,
                (long long)r1, (long long)lo, (long long)hi);
  if (r1 == r0) return KKM_OK;
  if (c->pc1 > 0) {  // a block: its c1 - c0 columns of each row
    const size_t w = (size_t)(c->pc1 - c->pc0) * 4;
    HIP_TRY(c, hipMemcpy2DAsync(out, w, (const float*)c->K + (r0 - c->pr0) * c->sz.ld, (size_t)c->sz.ld * 4, w,
                                (size_t)(r1 - r0), hipMemcpyDeviceToDevice, c->stream), "copy block rows");
    HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
    return KKM_OK;
  }
  if (c->mode == KKM_MODE_ONTHEFLY) {
    int rc = run(c, KKM_PHASE_OTHER, "kernel_rows", [&] {
      return launch_kernel_rows(c->Xp, c->nrm, c->maxnrm, c->sz.n, c->sz.d_pad, c->kp, r0, r1, out, c->stream);
    });
    if (rc) return rc;
    HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
    return KKM_OK;
  }
  if (c->mode == KKM_MODE_PACKED) {
    int rc = run(c, KKM_PHASE_OTHER, "packed_rows", [&] {
      return launch_packed_rows(c->K, c->storage == KKM_STORE_F16, c->kw, c->sz.n, c->sz.ld, r0, r1, out,
                                c->stream);
    });
    if (rc) return rc;
    HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
    return KKM_OK;
  }
  if (c->storage == KKM_STORE_F16) {
    int rc = run(c, KKM_PHASE_OTHER, "rows_f16", [&] {
      return launch_rows_f16((const half_t*)c->K, c->kw, c->sz.n, c->sz.ld, r0, r1, out, c->stream);
    });
    if (rc) return rc;
    HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
    return KKM_OK;
  }
  const size_t row = (size_t)c->sz.n * 4;
  HIP_TRY(c, hipMemcpy2DAsync(out, row, (const float*)c->K + r0 * c->sz.ld, (size_t)c->sz.ld * 4, row,
                              (size_t)(r1 - r0), hipMemcpyDeviceToDevice, c->stream), "copy rows");
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  return KKM_OK;
}

int kkm_copy_diag(kkm_ctx* c, float* out) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!c->built) return fail(c, KKM_ERR_STATE, "no kernel matrix built on this context");
  if (!out) return fail(c, KKM_ERR_ARG, "out is NULL");
  HIP_TRY(c, hipMemcpyAsync(out, c->diagK, (size_t)c->sz.n * 4, hipMemcpyDeviceToDevice, c->stream), "copy diag");
  HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
  return KKM_OK;
}

int kkm_set_timing(kkm_ctx* c, int32_t phase_mask) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  (void)hipStreamSynchronize(c->stream);
  collect_timing(c);
  c->timing = phase_mask & KKM_TIME_ALL;
  if (c->timing) c->tacc = kkm_timing{};
  return KKM_OK;
}

int kkm_get_timing(kkm_ctx* c, kkm_timing* out) {
  if (!c || !out) return fail(c, KKM_ERR_ARG, "NULL argument");
  collect_timing(c);
  *out = c->tacc;
  return KKM_OK;
}

int kkm_get_info(kkm_ctx* c, kkm_info* out) {
  if (!c || !out) return fail(c, KKM_ERR_ARG, "NULL argument");
  if (!c->built) return fail(c, KKM_ERR_STATE, "no kernel matrix built on this context");
  out->n = c->sz.n;
  out->d = c->d;
  out->d_pad = c->sz.d_pad;
  out->kind = c->kind;
  out->mode = c->mode;
  out->ld = c->sz.ld;
  out->storage = c->storage;
  out->bytes_K = k_bytes(c->wsz, c->mode, c->storage);
  out->bytes_total = c->held;
  if (c->fixups < 0) {
    unsigned long long cnt[kFixSegs] = {0};
    if (c->fix_count) {
      HIP_TRY(c, hipMemcpyAsync(cnt, c->fix_count, sizeof cnt, hipMemcpyDeviceToHost, c->stream), "read fix-up counts");
      HIP_TRY(c, hipStreamSynchronize(c->stream), "synchronize");
    }
    int64_t tot = 0;
    for (int q = 0; q < kFixSegs; ++q) tot += (int64_t)cnt[q];
    c->fixups = tot;
  }
  out->fixups = c->fixups;
  out->fixup_capacity = c->fix_cap;
  const bool blk = c->pc1 > 0;
  out->r0 = blk ? c->pr0 : 0;
  out->r1 = blk ? c->pr1 : c->sz.n;
  out->c0 = blk ? c->pc0 : 0;
  out->c1 = blk ? c->pc1 : c->sz.n;
  return KKM_OK;
}


// ---- achievable-peak microbenchmarks (measurement aids)

}  // extern "C"

namespace {

// Average duration of reps launches of `launch` on the context's stream,
// from one pair of HIP events around all of them.
template <class F>
int time_launches(kkm_ctx* c, int32_t reps, float* ms_out, F&& launch, const char* what) {
  hipEvent_t a = nullptr, b = nullptr;
  HIP_TRY(c, hipEventCreate(&a), "hipEventCreate");
  hipError_t e = hipEventCreate(&b);
  if (e != hipSuccess) {
    (void)hipEventDestroy(a);
    return hip_fail(c, e, "hipEventCreate");
  }
  e = hipEventRecord(a, c->stream);
  for (int32_t r = 0; r < reps && e == hipSuccess; ++r) e = launch();
  if (e == hipSuccess) e = hipEventRecord(b, c->stream);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  if (e != hipSuccess) return hip_fail(c, e, what);
  *ms_out = ms / (float)reps;
  return KKM_OK;
}

}  // namespace

extern "C" {

int kkm_peak_read(kkm_ctx* c, const void* buf, size_t bytes, float* sums, int32_t reps, float* ms_out) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!buf || !sums || !ms_out) return fail(c, KKM_ERR_ARG, "NULL argument");
  if (bytes < 16 || bytes % 16 || (uintptr_t)buf % 16) return fail(c, KKM_ERR_ARG, "bytes=%zu must be a positive multiple of 16 on a 16-byte aligned buffer", bytes);
  if (reps < 1) return fail(c, KKM_ERR_ARG, "reps=%d must be >= 1", reps);
  return time_launches(c, reps, ms_out, [&] { return launch_peak_read(buf, (int64_t)bytes, sums, c->stream); },
                       "peak read");
}

int kkm_peak_write(kkm_ctx* c, void* buf, size_t bytes, float value, int32_t reps, float* ms_out) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!buf || !ms_out) return fail(c, KKM_ERR_ARG, "NULL argument");
  if (bytes < 16 || bytes % 16 || (uintptr_t)buf % 16) return fail(c, KKM_ERR_ARG, "bytes=%zu must be a positive multiple of 16 on a 16-byte aligned buffer", bytes);
  if (reps < 1) return fail(c, KKM_ERR_ARG, "reps=%d must be >= 1", reps);
  return time_launches(c, reps, ms_out, [&] { return launch_peak_write(buf, (int64_t)bytes, value, c->stream); },
                       "peak write");
}

int kkm_peak_read_rows(kkm_ctx* c, const void* buf, int64_t nrows, int64_t ld, const int32_t* rows, int32_t nchunks,
                       int32_t seg, float* sums, int32_t reps, float* ms_out) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!buf || !rows || !sums || !ms_out) return fail(c, KKM_ERR_ARG, "NULL argument");
  if ((uintptr_t)buf % 16) return fail(c, KKM_ERR_ARG, "buf must be 16-byte aligned");
  if (nrows < 1 || ld < 128 || ld % 4) return fail(c, KKM_ERR_ARG, "nrows=%lld must be >= 1 and ld=%lld a multiple of 4, >= 128", (long long)nrows, (long long)ld);
  if (seg < 128 || seg % 128 || seg > ld) return fail(c, KKM_ERR_ARG, "seg=%d must be a positive multiple of 128, at most ld", seg);
  // the launch's work-items (512 per workgroup) must fit the 32-bit grid
  if (nchunks < 1 || (int64_t)nchunks * (ld / seg) * 512 > (int64_t)UINT32_MAX)
    return fail(c, KKM_ERR_ARG, "nchunks=%d x %lld segments is out of range", nchunks, (long long)(ld / seg));
  if (reps < 1) return fail(c, KKM_ERR_ARG, "reps=%d must be >= 1", reps);
  return time_launches(c, reps, ms_out, [&] {
        return launch_peak_rows((const float*)buf, nrows, ld, rows, nchunks, seg, sums, c->stream);
      }, "peak rows");
}

int kkm_peak_mfma(kkm_ctx* c, int32_t iters, float* out, int32_t reps, float* ms_out, double* flops_out) {
  if (!c) return fail(nullptr, KKM_ERR_ARG, "ctx is NULL");
  if (!out || !ms_out || !flops_out) return fail(c, KKM_ERR_ARG, "NULL argument");
  if (iters < 1 || reps < 1) return fail(c, KKM_ERR_ARG, "iters=%d and reps=%d must be >= 1", iters, reps);
  *flops_out = (double)kPeakMfmaGrid * 4.0 * 4.0 * 4096.0 * (double)iters;
  return time_launches(c, reps, ms_out, [&] { return launch_peak_mfma(iters, out, c->stream); }, "peak mfma");
}

}  // extern "C"
