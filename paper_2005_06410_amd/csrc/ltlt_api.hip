// Host side of the C ABI declared in include/ltlt.h: argument checks, the
// per-device workspace, the block loop of the factorization and optional
// per-kernel event timing.  Every compute step runs in the gfx950 kernels of
// this library; nothing here touches matrix data on the host.

#include <algorithm>
#include <atomic>
#include <map>
#include <mutex>
#include <utility>
#include <vector>

#include "ltlt.h"
#include "ltlt_internal.h"

using namespace ltlt;

namespace {

constexpr int kDefaultNb = 128;
constexpr int kMinFallbackNb = 32;       // narrowest width ltlt_factor falls back to
constexpr int kDefaultComplexNb = 128;          // complex: 32 register slots per lane, four lanes per row
constexpr int kMaxComplexNb = 128;
constexpr int64_t kMaxOrder = (1 << 21) - 1;   // exchange records pack indices in 21 bits
constexpr size_t kLdsBudget = 160 * 1024 - 2048;   // dynamic LDS a panel workgroup may use

int hip_err(hipError_t e) { return LTLT_ERR_HIP_BASE - (int)e; }

// ---- fixed per-device array: status words and the allocation-free workspace --
// `scratch` is a file-scope device array: every GPU the library runs on holds
// its own copy, at its own address, until the process ends.  Its first 256
// bytes are the two bounded-wait status words of every call on that device
// (see raise_wait_status); the rest is the whole workspace of
// ltlt_factor_noalloc, which therefore needs no allocation.  In host code the
// name `scratch` is only a stand-in for the symbol: its device address on the
// current device comes from hipGetSymbolAddress, looked up once per device and
// kept in g_scratch_ptr, and only that address is ever handed to kernels.
constexpr size_t kScratchBytes = (size_t)16 << 20;
constexpr size_t kScratchStatusBytes = 256;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxScratchDevices] = {};   // fixed table: no host allocation either

__global__ void zero_words_kernel(int* p, int count) {
  const int i = threadIdx.x;
  if (i < count) p[i] = 0;
}

// Device address of `scratch` on the current device.  The first call on a
// device looks it up and clears the status words with a kernel on `s`
// (stream-ordered before the caller's kernels).
hipError_t device_scratch(hipStream_t s, char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(zero_words_kernel, dim3(1), dim3(64), 0, s, static_cast<int*>(p),
                       (int)(kScratchStatusBytes / sizeof(int)));
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

// The status words of the current device (set up on first use).
hipError_t status_words(hipStream_t s, int** status) {
  char* base = nullptr;
  const hipError_t e = device_scratch(s, &base);
  if (e == hipSuccess) *status = reinterpret_cast<int*>(base);
  return e;
}

// ---- per-device workspace (grown on demand) ---------------------------------
struct Workspace {
  void* ptr = nullptr;
  size_t bytes = 0;
};
std::mutex g_ws_mu;
std::map<int, Workspace> g_ws;

// A caller-provided workspace (the allocation-free entry point).
struct FixedWs {
  char* ptr;
  size_t bytes;
  int* status;
};

hipError_t workspace(size_t bytes, hipStream_t s, void** out, int** status) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = status_words(s, status);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  Workspace& w = g_ws[dev];
  if (w.bytes < bytes) {
    if (w.ptr) {
      e = hipDeviceSynchronize();       // earlier work may still use it
      if (e != hipSuccess) return e;
      e = hipFree(w.ptr);
      if (e != hipSuccess) return e;
      w.ptr = nullptr;
      w.bytes = 0;
    }
    size_t want = std::max(bytes, (size_t)1 << 20);
    e = hipMalloc(&w.ptr, want);
    if (e != hipSuccess) { w.ptr = nullptr; return e; }
    w.bytes = want;
  }
  *out = w.ptr;
  return hipSuccess;
}

// bump allocator inside the workspace (256-byte aligned pieces)
struct Carve {
  size_t off = 0;
  template <typename U> size_t take(size_t count) {
    size_t at = off;
    off += (count * sizeof(U) + 255) & ~(size_t)255;
    return at;
  }
};

}  // namespace

namespace ltlt {
namespace {
std::atomic<bool> g_cooperative_panels{false};
std::atomic<bool> g_forced_timeout{false};
}  // namespace
bool cooperative_panels() { return g_cooperative_panels.load(std::memory_order_relaxed); }
bool forced_timeout() { return g_forced_timeout.load(std::memory_order_relaxed); }

hipError_t ensure_dynamic_lds(const void* kernel, int bytes) {
  // a fixed table of (kernel, device) -> bytes allowed: no host allocation, so
  // the allocation-free entry point may pass through here
  struct Entry { const void* kernel; int dev; int bytes; };
  constexpr int kEntries = 256;
  static Entry table[kEntries];
  static int used = 0;
  static std::mutex mu;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(mu);
  int at = -1;
  for (int i = 0; i < used; ++i)
    if (table[i].kernel == kernel && table[i].dev == dev) { at = i; break; }
  if (at >= 0 && table[at].bytes >= bytes) return hipSuccess;
  e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  if (at < 0 && used < kEntries) at = used++;
  if (at >= 0) table[at] = Entry{kernel, dev, bytes};   // a full table only means setting it again
  return hipSuccess;
}
}  // namespace ltlt

namespace {

// ---- profiling ---------------------------------------------------------------
// Per-launch timing with HIP events on the launch stream.  The events only
// time: they are created without the system-scope fence that a default
// event record performs (an L2 writeback and invalidate at every record,
// which cost about 3 ms per n = 16384 factorization), and they are reused
// from a per-device pool instead of being created for every launch.
struct ProfRec {
  int kind;
  int dev;
  hipEvent_t a, b;
  double flops;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
bool g_prof_update_only = false;                      // record the trailing updates alone
std::vector<ProfRec> g_prof;
std::map<int, std::vector<hipEvent_t>> g_event_pool;   // by device

bool take_event_locked(int dev, hipEvent_t* ev) {
  auto& pool = g_event_pool[dev];
  if (!pool.empty()) { *ev = pool.back(); pool.pop_back(); return true; }
  return hipEventCreateWithFlags(ev, hipEventDisableSystemFence) == hipSuccess;
}

struct ProfScope {
  ProfRec rec{};
  bool on = false;
  hipStream_t s;
  // kind < 0: never recorded (the allocation-free path creates no events)
  ProfScope(int kind, double flops, hipStream_t st) : s(st) {
    if (kind < 0) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (!g_prof_on || (g_prof_update_only && kind != 1)) return;
    rec.kind = kind;
    rec.flops = flops;
    if (hipGetDevice(&rec.dev) != hipSuccess) return;
    if (!take_event_locked(rec.dev, &rec.a)) return;
    if (!take_event_locked(rec.dev, &rec.b)) { g_event_pool[rec.dev].push_back(rec.a); return; }
    on = (hipEventRecord(rec.a, s) == hipSuccess);
    if (!on) { g_event_pool[rec.dev].push_back(rec.a); g_event_pool[rec.dev].push_back(rec.b); }
  }
  ~ProfScope() {
    if (!on) return;
    (void)hipEventRecord(rec.b, s);
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof.push_back(rec);
  }
};

// Records are dropped and their events go back to the pool (a recorded
// event may be recorded again once the caller has synchronized, which it has
// whenever it reads or restarts the profile).
void prof_clear_locked() {
  for (auto& r : g_prof) {
    g_event_pool[r.dev].push_back(r.a);
    g_event_pool[r.dev].push_back(r.b);
  }
  g_prof.clear();
}

// ---- factorization -----------------------------------------------------------
template <typename T>
int choose_rows(int bw) {
  const int R = panel_rows(bw);
  return panel_lds_bytes<T>(bw, R) <= kLdsBudget ? R : 0;
}

// fixed == nullptr: the cached, grown-on-demand workspace; otherwise the
// caller's fixed one (LTLT_ERR_SCRATCH when the order needs more), with no
// allocation and no profiling events.
template <typename T>
int factor_impl(int64_t n64, T* A, int64_t lda, int32_t* ipiv, int nb, hipStream_t s,
                const FixedWs* fixed = nullptr) {
  if (n64 == 0) return 0;
  if (n64 >= kMaxOrder) return LTLT_ERR_UNSUPPORTED;
  const int n = (int)n64;
  const int nsteps = std::max(n - 2, 0);
  const int nblk = nsteps > 0 ? (nsteps + nb - 1) / nb : 0;
  const int bw0 = std::min(nb, std::max(nsteps, 1));

  // panel geometry of the largest block (block 0) bounds every other block
  const int R = choose_rows<T>(bw0);
  int Pmax = 1;
  if (nblk > 0) {
    if (R == 0) return LTLT_ERR_UNSUPPORTED;
    const size_t lds = panel_lds_bytes<T>(bw0, R);
    Pmax = (n - 1 + R - 1) / R;
    const int cap = panel_max_blocks<T>(bw0, lds);
    if (cap <= 0 || Pmax > cap) return LTLT_ERR_UNSUPPORTED;
  }

  const int64_t ldw = ((int64_t)n + 63) / 64 * 64;
  const int c_end = nblk >= 2 ? (nblk - 1) * nb : 0;
  Carve cv;
  const size_t o_PO = cv.take<T>((size_t)ldw * (nb + 1));
  const size_t o_Bm = cv.take<T>((size_t)ldw * (nb + 1));
  const size_t o_G = cv.take<T>((size_t)ldw * nb);
  const size_t o_al = cv.take<T>((size_t)nb);
  const size_t o_T = cv.take<int>((size_t)std::max(nblk, 1) * n);
  const size_t o_GC = cv.take<int>((size_t)std::max(nblk, 1) * n);
  const int nrec = Pmax;                      // exchange records per slot
  const size_t o_rec = cv.take<uint64_t>((size_t)2 * kRecStride * nrec);
  const size_t o_st = cv.take<T>(perm_stage_elems<T>(n, c_end));

  void* ws = nullptr;
  int* status = nullptr;
  hipError_t e = hipSuccess;
  if (fixed) {
    if (cv.off > fixed->bytes) return LTLT_ERR_SCRATCH;
    ws = fixed->ptr;
    status = fixed->status;
  } else {
    e = workspace(cv.off, s, &ws, &status);
    if (e != hipSuccess) return hip_err(e);
  }
  const int pk = fixed ? -1 : 0;                 // profiling kinds are offset by this (-1: off)
  char* base = static_cast<char*>(ws);
  T* PO = reinterpret_cast<T*>(base + o_PO);
  T* Bm = reinterpret_cast<T*>(base + o_Bm);
  T* Gm = reinterpret_cast<T*>(base + o_G);
  T* al = reinterpret_cast<T*>(base + o_al);
  int* Tblk = reinterpret_cast<int*>(base + o_T);
  int* Gc = reinterpret_cast<int*>(base + o_GC);
  uint64_t* rec = reinterpret_cast<uint64_t*>(base + o_rec);
  T* stage = reinterpret_cast<T*>(base + o_st);

  {
    ProfScope ps(pk < 0 ? -1 : 3, 0.0, s);
    e = launch_init(ipiv, n, status, s);
    if (e == hipSuccess && nblk > 0) e = launch_rec_init(rec, nrec, s);
  }
  if (e != hipSuccess) return hip_err(e);

  for (int J = 0; J < nblk; ++J) {
    const int j = J * nb;
    const int bw = std::min(nb, nsteps - j);
    const int m = n - j - 1;
    PanelArgs pa{};
    pa.A = A; pa.lda = lda; pa.n = n; pa.j = j; pa.bw = bw;
    pa.R = choose_rows<T>(bw);
    pa.P = (m + pa.R - 1) / pa.R;
    pa.nrec = nrec;
    pa.G = Gm; pa.PO = PO; pa.Bm = Bm; pa.ldw = ldw; pa.alpha = al;
    pa.perm = Tblk + (int64_t)J * n;
    pa.ipiv = ipiv;
    pa.rec = rec;
    pa.status = status;
    {
      ProfScope ps(pk < 0 ? -1 : 0, 0.0, s);
      e = launch_panel<T>(pa, panel_lds_bytes<T>(bw, pa.R), s);
    }
    if (e != hipSuccess) return hip_err(e);

    const int i0 = j + bw + 1;
    const int m2 = n - i0;
    if (m2 >= 2) {
      UpdateArgs ua{};
      ua.C = A + (int64_t)i0 + (int64_t)i0 * lda;
      ua.ldc = lda;
      ua.m = m2;
      ua.perm = Tblk + (int64_t)J * n + i0;
      ua.perm_base = i0;
      ua.perm_lo = (j + 1) - i0;     // rows held since block start: j+1 .. n-1
      ua.perm_hi = m2 - 1;
      ua.K = bw + 1;
      ua.Lx = PO + bw;
      ua.ldl = ldw;
      ua.Bt = Bm;
      ua.ldb = ldw;
      ua.pad_row = 1;      // bw + m2 + 1 <= n <= ldw: row m2 of each column lies inside the workspace
      ProfScope ps(pk < 0 ? -1 : 1, (double)m2 * (double)m2 * (double)bw, s);
      e = launch_update<T>(ua, s);
      if (e != hipSuccess) return hip_err(e);
    }
    {
      ProfScope ps(pk < 0 ? -1 : 2, 0.0, s);
      e = launch_commit<T>(A, lda, n, j, bw, PO, ldw, al, status, s);
    }
    if (e != hipSuccess) return hip_err(e);
  }

  if (nblk >= 2) {
    ProfScope ps(pk < 0 ? -1 : 3, 0.0, s);
    e = launch_perm_chain(Tblk, nb, nblk, n, Gc, s);
    if (e == hipSuccess) e = launch_perm_apply<T>(A, lda, n, Gc, nb, c_end, stage, s);
    if (e != hipSuccess) return hip_err(e);
  }
  return 0;
}

// Pfaffian by the even column steps only (see ltlt_pair.hip): blocks of nb
// columns, nb/2 steps each; every block is a pair panel, a rank-nb trailing
// update of positions >= j+nb (no carry column), then the block's alphas into
// A(k+1, k).  The Pfaffian is read off at the end from those alphas and the
// pivots, by the same kernel as for the full factorization.
template <typename T>
int pfaffian_direct_impl(int64_t n64, T* A, int64_t lda, int32_t* ipiv, int nb, double* logabs, int32_t* sign,
                         hipStream_t s) {
  if (n64 >= kMaxOrder) return LTLT_ERR_UNSUPPORTED;
  const int n = (int)n64;
  hipError_t e = hipSuccess;
  if (n == 0 || (n & 1)) {                       // Pf = 1 (n = 0) or 0 (odd n): no steps
    void* ws = nullptr;
    int* status = nullptr;
    e = workspace(256, s, &ws, &status);
    if (e == hipSuccess && n > 0) e = launch_init(ipiv, n, status, s);
    if (e == hipSuccess) e = launch_pfaffian<T>(n, A, lda, ipiv, logabs, sign, status, s);
    return e == hipSuccess ? 0 : hip_err(e);
  }
  const int bw0 = std::min(nb, n);
  const int R = pair_panel_rows(bw0);
  if (pair_lds_bytes<T>(bw0, R) > kLdsBudget) return LTLT_ERR_UNSUPPORTED;
  const int Pmax = (n - 1 + R - 1) / R;
  const int cap = pair_max_blocks<T>(bw0, pair_lds_bytes<T>(bw0, R));
  if (cap <= 0 || Pmax > cap) return LTLT_ERR_UNSUPPORTED;

  const int64_t ldw = ((int64_t)n + 63) / 64 * 64;
  Carve cv;
  const size_t o_PO = cv.take<T>((size_t)ldw * nb);
  const size_t o_Bm = cv.take<T>((size_t)ldw * nb);
  const size_t o_G = cv.take<T>((size_t)ldw * nb);
  const size_t o_al = cv.take<T>((size_t)nb);
  const size_t o_T = cv.take<int>((size_t)n);
  const int nrec = Pmax;
  const size_t o_rec = cv.take<uint64_t>((size_t)2 * kRecStride * nrec);
  void* ws = nullptr;
  int* status = nullptr;
  e = workspace(cv.off, s, &ws, &status);
  if (e != hipSuccess) return hip_err(e);
  char* base = static_cast<char*>(ws);
  T* PO = reinterpret_cast<T*>(base + o_PO);
  T* Bm = reinterpret_cast<T*>(base + o_Bm);
  T* Gm = reinterpret_cast<T*>(base + o_G);
  T* al = reinterpret_cast<T*>(base + o_al);
  int* Tperm = reinterpret_cast<int*>(base + o_T);
  uint64_t* rec = reinterpret_cast<uint64_t*>(base + o_rec);
  {
    ProfScope ps(3, 0.0, s);
    e = launch_init(ipiv, n, status, s);
    if (e == hipSuccess) e = launch_rec_init(rec, nrec, s);
  }
  if (e != hipSuccess) return hip_err(e);

  for (int j = 0; j < n; j += nb) {
    const int bw = std::min(nb, n - j);          // even: n and nb are
    const int m = n - j - 1;                     // rows at positions j+1 .. n-1
    PanelArgs pa{};
    pa.A = A; pa.lda = lda; pa.n = n; pa.j = j; pa.bw = bw;
    pa.R = pair_panel_rows(bw);
    pa.P = (m + pa.R - 1) / pa.R;
    pa.nrec = nrec;
    pa.G = Gm; pa.PO = PO; pa.Bm = Bm; pa.ldw = ldw; pa.alpha = al;
    pa.perm = Tperm;
    pa.ipiv = ipiv;
    pa.rec = rec;
    pa.status = status;
    {
      ProfScope ps(0, 0.0, s);
      e = launch_pair_panel<T>(pa, pair_lds_bytes<T>(bw, pa.R), s);
    }
    if (e != hipSuccess) return hip_err(e);
    const int i0 = j + bw;
    const int m2 = n - i0;
    if (m2 >= 2) {
      UpdateArgs ua{};
      ua.C = A + (int64_t)i0 + (int64_t)i0 * lda;
      ua.ldc = lda;
      ua.m = m2;
      ua.perm = Tperm + i0;
      ua.perm_base = i0;
      ua.perm_lo = (j + 1) - i0;
      ua.perm_hi = m2 - 1;
      ua.K = bw;
      ua.Lx = PO;
      ua.ldl = ldw;
      ua.Bt = Bm;
      ua.ldb = ldw;
      ua.pad_row = 1;      // m2 < n <= ldw: row m2 of each column lies inside the workspace
      ProfScope ps(1, (double)m2 * (double)m2 * (double)bw, s);
      e = launch_update<T>(ua, s);
      if (e != hipSuccess) return hip_err(e);
    }
    {
      ProfScope ps(2, 0.0, s);
      e = launch_pair_commit<T>(A, lda, j, bw / 2, al, status, s);
    }
    if (e != hipSuccess) return hip_err(e);
  }
  {
    ProfScope ps(3, 0.0, s);
    e = launch_pfaffian<T>(n, A, lda, ipiv, logabs, sign, status, s);
  }
  return e == hipSuccess ? 0 : hip_err(e);
}

bool bad_dtype(int d) { return d != LTLT_F64 && d != LTLT_F32; }
bool is_complex(int d) { return d == LTLT_C128 || d == LTLT_C64; }

// Complex factorization: X is split into real and imaginary planes
// (workspace, leading dimension ldw), every block runs the complex panel,
// then each plane's trailing update as one real product of depth 2(bw+1)
// (Re C += [Lr Li][Btr -Bti]^T, Im C += [Li Lr][Btr Bti]^T) with the real
// update kernel, and the per-plane commit; the final row order is applied to
// each plane and the planes are merged back into A.  T is the component type.
template <typename T>
int factor_complex_impl(int64_t n64, void* A, int64_t lda, int32_t* ipiv, int nb, hipStream_t s) {
  if (n64 == 0) return 0;
  if (n64 >= kMaxOrder) return LTLT_ERR_UNSUPPORTED;
  const int n = (int)n64;
  const int nsteps = std::max(n - 2, 0);
  const int nblk = nsteps > 0 ? (nsteps + nb - 1) / nb : 0;
  const int bw0 = std::min(nb, std::max(nsteps, 1));
  const int R = cpanel_rows(bw0);
  int Pmax = 1;
  if (nblk > 0) {
    const size_t lds = cpanel_lds_bytes<T>(bw0);
    if (lds > kLdsBudget) return LTLT_ERR_UNSUPPORTED;
    Pmax = (n - 1 + R - 1) / R;
    const int cap = cpanel_max_blocks<T>(bw0, lds);
    if (cap <= 0 || Pmax > cap) return LTLT_ERR_UNSUPPORTED;
  }

  const int64_t ldw = ((int64_t)n + 63) / 64 * 64;
  const int K0 = nb + 1;
  const int c_end = nblk >= 2 ? (nblk - 1) * nb : 0;
  Carve cv;
  const size_t o_Pr = cv.take<T>((size_t)ldw * n);
  const size_t o_Pi = cv.take<T>((size_t)ldw * n);
  const size_t o_LL = cv.take<T>((size_t)ldw * 3 * K0);
  const size_t o_BA = cv.take<T>((size_t)ldw * 2 * K0);
  const size_t o_BB = cv.take<T>((size_t)ldw * 2 * K0);
  const size_t o_Gr = cv.take<T>((size_t)ldw * nb);
  const size_t o_Gi = cv.take<T>((size_t)ldw * nb);
  const size_t o_Vr = cv.take<T>((size_t)ldw);
  const size_t o_Vi = cv.take<T>((size_t)ldw);
  const size_t o_ar = cv.take<T>((size_t)nb);
  const size_t o_ai = cv.take<T>((size_t)nb);
  const size_t o_T = cv.take<int>((size_t)std::max(nblk, 1) * n);
  const size_t o_GC = cv.take<int>((size_t)std::max(nblk, 1) * n);
  const int nrec = Pmax;
  const size_t o_rec = cv.take<uint64_t>((size_t)2 * kRecStride * nrec);
  const size_t o_st = cv.take<T>(perm_stage_elems<T>(n, c_end));

  void* ws = nullptr;
  int* status = nullptr;
  hipError_t e = workspace(cv.off, s, &ws, &status);
  if (e != hipSuccess) return hip_err(e);
  char* base = static_cast<char*>(ws);
  T* Pr = reinterpret_cast<T*>(base + o_Pr);
  T* Pi = reinterpret_cast<T*>(base + o_Pi);
  T* LL = reinterpret_cast<T*>(base + o_LL);
  T* BA = reinterpret_cast<T*>(base + o_BA);
  T* BB = reinterpret_cast<T*>(base + o_BB);
  T* Gr = reinterpret_cast<T*>(base + o_Gr);
  T* Gi = reinterpret_cast<T*>(base + o_Gi);
  T* Vr = reinterpret_cast<T*>(base + o_Vr);
  T* Vi = reinterpret_cast<T*>(base + o_Vi);
  T* alr = reinterpret_cast<T*>(base + o_ar);
  T* ali = reinterpret_cast<T*>(base + o_ai);
  int* Tblk = reinterpret_cast<int*>(base + o_T);
  int* Gc = reinterpret_cast<int*>(base + o_GC);
  uint64_t* rec = reinterpret_cast<uint64_t*>(base + o_rec);
  T* stage = reinterpret_cast<T*>(base + o_st);

  {
    ProfScope ps(3, 0.0, s);
    e = launch_init(ipiv, n, status, s);
    if (e == hipSuccess && nblk > 0) e = launch_rec_init(rec, nrec, s);
    if (e == hipSuccess) e = launch_cplx_split<T>(n, A, lda, Pr, Pi, ldw, s);
  }
  if (e != hipSuccess) return hip_err(e);

  for (int J = 0; J < nblk; ++J) {
    const int j = J * nb;
    const int bw = std::min(nb, nsteps - j);
    const int K = bw + 1;
    const int m = n - j - 1;
    CPanelArgs ca{};
    PanelArgs& pa = ca.b;
    pa.A = Pr; pa.lda = ldw; pa.n = n; pa.j = j; pa.bw = bw;
    pa.R = cpanel_rows(bw);
    pa.P = (m + pa.R - 1) / pa.R;
    pa.nrec = nrec;
    pa.G = Gr; pa.ldw = ldw; pa.alpha = alr;
    pa.perm = Tblk + (int64_t)J * n;
    pa.ipiv = ipiv;
    pa.rec = rec;
    pa.status = status;
    ca.Ai = Pi; ca.Gi = Gi; ca.Vr = Vr; ca.Vi = Vi;
    ca.LL = LL; ca.BtA = BA; ca.BtB = BB; ca.alpha_i = ali;
    {
      ProfScope ps(0, 0.0, s);
      e = launch_cpanel<T>(ca, cpanel_lds_bytes<T>(bw), s);
    }
    if (e != hipSuccess) return hip_err(e);

    const int i0 = j + bw + 1;
    const int m2 = n - i0;
    if (m2 >= 2) {
      for (int plane = 0; plane < 2; ++plane) {
        UpdateArgs ua{};
        ua.C = (plane == 0 ? Pr : Pi) + (int64_t)i0 + (int64_t)i0 * ldw;
        ua.ldc = ldw;
        ua.m = m2;
        ua.perm = Tblk + (int64_t)J * n + i0;
        ua.perm_base = i0;
        ua.perm_lo = (j + 1) - i0;
        ua.perm_hi = m2 - 1;
        ua.K = 2 * K;
        ua.Lx = LL + (plane == 0 ? 0 : (int64_t)K * ldw) + bw;
        ua.ldl = ldw;
        ua.Bt = plane == 0 ? BA : BB;
        ua.ldb = ldw;
        ua.pad_row = 1;    // row bw + m2 = n - j - 1 < ldw of every operand column lies inside its column
        ProfScope ps(1, 2.0 * (double)m2 * (double)m2 * (double)bw, s);   // depth 2 bw: half the complex work
        e = launch_update<T>(ua, s);
        if (e != hipSuccess) return hip_err(e);
      }
    }
    {
      ProfScope ps(2, 0.0, s);
      e = launch_commit<T>(Pr, ldw, n, j, bw, LL, ldw, alr, status, s);
      if (e == hipSuccess) e = launch_commit<T>(Pi, ldw, n, j, bw, LL + (int64_t)K * ldw, ldw, ali, status, s);
    }
    if (e != hipSuccess) return hip_err(e);
  }

  {
    ProfScope ps(3, 0.0, s);
    if (nblk >= 2) {
      e = launch_perm_chain(Tblk, nb, nblk, n, Gc, s);
      if (e == hipSuccess) e = launch_perm_apply<T>(Pr, ldw, n, Gc, nb, c_end, stage, s);
      if (e == hipSuccess) e = launch_perm_apply<T>(Pi, ldw, n, Gc, nb, c_end, stage, s);
    }
    if (e == hipSuccess) e = launch_cplx_merge<T>(n, A, lda, Pr, Pi, ldw, s);
  }
  return e == hipSuccess ? 0 : hip_err(e);
}

}  // namespace

extern "C" {

int ltlt_factor_nb(int64_t n, void* A, int64_t lda, int dtype, int32_t* ipiv, int nb, hipStream_t stream) {
  if (n < 0 || n > (int64_t)INT32_MAX / 2) return -1;
  if (A == nullptr && n > 0) return -2;
  if (lda < std::max<int64_t>(1, n)) return -3;
  if (bad_dtype(dtype) && !is_complex(dtype)) return -4;
  if (ipiv == nullptr && n > 0) return -5;
  if (nb < 1 || nb > (is_complex(dtype) ? kMaxComplexNb : kMaxNb)) return -6;
  if (n == 0) return 0;
  if (dtype == LTLT_C128) return factor_complex_impl<double>(n, A, lda, ipiv, (int)nb, stream);
  if (dtype == LTLT_C64) return factor_complex_impl<float>(n, A, lda, ipiv, (int)nb, stream);
  if (dtype == LTLT_F64) return factor_impl<double>(n, static_cast<double*>(A), lda, ipiv, (int)nb, stream);
  return factor_impl<float>(n, static_cast<float*>(A), lda, ipiv, (int)nb, stream);
}

int ltlt_factor(int64_t n, void* A, int64_t lda, int dtype, int32_t* ipiv, hipStream_t stream) {
  // The panel holds every row of the block in registers of co-resident
  // workgroups; narrower blocks fit more rows per workgroup.  When the default
  // width needs more workgroups than the device holds, halve it (the size
  // checks come before any allocation or launch, so a refused width leaves
  // nothing behind).
  int nb = is_complex(dtype) ? kDefaultComplexNb : kDefaultNb;
  int r = ltlt_factor_nb(n, A, lda, dtype, ipiv, nb, stream);
  while (r == LTLT_ERR_UNSUPPORTED && nb > kMinFallbackNb && n < kMaxOrder) {
    nb /= 2;
    r = ltlt_factor_nb(n, A, lda, dtype, ipiv, nb, stream);
  }
  return r;
}

int ltlt_factor_noalloc(int64_t n, void* A, int64_t lda, int dtype, int32_t* ipiv, hipStream_t stream) {
  if (n < 0 || n > (int64_t)INT32_MAX / 2) return -1;
  if (A == nullptr && n > 0) return -2;
  if (lda < std::max<int64_t>(1, n)) return -3;
  if (bad_dtype(dtype)) return -4;              // real types only (complex needs 2 n^2 of planes)
  if (ipiv == nullptr && n > 0) return -5;
  if (n == 0) return 0;
  char* base = nullptr;
  const hipError_t e = device_scratch(stream, &base);
  if (e != hipSuccess) return hip_err(e);
  const FixedWs fw{base + kScratchStatusBytes, kScratchBytes - kScratchStatusBytes, reinterpret_cast<int*>(base)};
  if (dtype == LTLT_F64)
    return factor_impl<double>(n, static_cast<double*>(A), lda, ipiv, kDefaultNb, stream, &fw);
  return factor_impl<float>(n, static_cast<float*>(A), lda, ipiv, kDefaultNb, stream, &fw);
}

int ltlt_pfaffian_complex(int64_t n, const void* A, int64_t lda, int dtype, const int32_t* ipiv, double* logabs,
                          double* phase, hipStream_t stream) {
  if (n < 0 || n > (int64_t)INT32_MAX / 2) return -1;
  if (A == nullptr && n > 0) return -2;
  if (lda < std::max<int64_t>(1, n)) return -3;
  if (!is_complex(dtype)) return -4;
  if (ipiv == nullptr && n > 0) return -5;
  if (logabs == nullptr) return -6;
  if (phase == nullptr) return -7;
  int* status = nullptr;
  hipError_t e = status_words(stream, &status);
  if (e != hipSuccess) return hip_err(e);
  e = dtype == LTLT_C128 ? launch_cpfaffian<double>((int)n, A, lda, ipiv, logabs, phase, status, stream)
                         : launch_cpfaffian<float>((int)n, A, lda, ipiv, logabs, phase, status, stream);
  return e == hipSuccess ? 0 : hip_err(e);
}

int ltlt_pfaffian(int64_t n, const void* A, int64_t lda, int dtype, const int32_t* ipiv, double* logabs,
                  int32_t* sign, hipStream_t stream) {
  if (n < 0 || n > (int64_t)INT32_MAX / 2) return -1;
  if (A == nullptr && n > 0) return -2;
  if (lda < std::max<int64_t>(1, n)) return -3;
  if (bad_dtype(dtype)) return -4;
  if (ipiv == nullptr && n > 0) return -5;
  if (logabs == nullptr) return -6;
  if (sign == nullptr) return -7;
  int* status = nullptr;
  hipError_t e = status_words(stream, &status);
  if (e != hipSuccess) return hip_err(e);
  if (dtype == LTLT_F64)
    e = launch_pfaffian<double>((int)n, static_cast<const double*>(A), lda, ipiv, logabs, sign, status, stream);
  else
    e = launch_pfaffian<float>((int)n, static_cast<const float*>(A), lda, ipiv, logabs, sign, status, stream);
  return e == hipSuccess ? 0 : hip_err(e);
}

int ltlt_pfaffian_direct(int64_t n, void* A, int64_t lda, int dtype, int32_t* ipiv, int nb, double* logabs,
                         int32_t* sign, hipStream_t stream) {
  if (n < 0 || n > (int64_t)INT32_MAX / 2) return -1;
  if (A == nullptr && n > 0) return -2;
  if (lda < std::max<int64_t>(1, n)) return -3;
  if (bad_dtype(dtype)) return -4;
  if (ipiv == nullptr && n > 0) return -5;
  const bool default_width = nb == 0;
  if (default_width) nb = kDefaultNb;
  if (nb < 2 || nb > kMaxNb || (nb & 1)) return -6;
  if (logabs == nullptr) return -7;
  if (sign == nullptr) return -8;
  auto run = [&](int w) {
    return dtype == LTLT_F64
               ? pfaffian_direct_impl<double>(n, static_cast<double*>(A), lda, ipiv, (int)w, logabs, sign, stream)
               : pfaffian_direct_impl<float>(n, static_cast<float*>(A), lda, ipiv, (int)w, logabs, sign, stream);
  };
  int r = run(nb);
  // as ltlt_factor: a default width whose pair panel does not fit is halved
  // (the size checks precede any launch)
  while (default_width && r == LTLT_ERR_UNSUPPORTED && nb > kMinFallbackNb && n < kMaxOrder) {
    nb /= 2;
    r = run(nb);
  }
  return r;
}

int ltlt_solve(int64_t n, const void* A, int64_t lda, int dtype, const int32_t* ipiv, int64_t nrhs, void* B,
               int64_t ldb, hipStream_t stream) {
  if (n < 0 || n > (int64_t)INT32_MAX / 2) return -1;
  if (A == nullptr && n > 0) return -2;
  if (lda < std::max<int64_t>(1, n)) return -3;
  if (bad_dtype(dtype)) return -4;
  if (ipiv == nullptr && n > 0) return -5;
  if (nrhs < 0 || nrhs > (int64_t)INT32_MAX / 2) return -6;
  if (B == nullptr && n > 0 && nrhs > 0) return -7;
  if (ldb < std::max<int64_t>(1, n)) return -8;
  if (n & 1) return LTLT_ERR_SINGULAR;           // a skew matrix of odd order is singular
  if (n == 0 || nrhs == 0) return 0;
  const size_t esz = dtype == LTLT_F64 ? sizeof(double) : sizeof(float);
  const int64_t ldy = (n + 63) / 64 * 64;
  const int nblk = (int)((n + 63) / 64);
  Carve cv;
  const size_t o_perm = cv.take<int>((size_t)n);
  const size_t o_cnt = cv.take<int>((size_t)2 * n);
  const size_t o_off = cv.take<int>((size_t)n + 1);
  const size_t o_list = cv.take<int>((size_t)n);
  const size_t o_al = cv.take<char>((size_t)n * esz);
  const size_t o_ral = cv.take<char>((size_t)n * esz);
  const size_t o_Y = cv.take<char>((size_t)ldy * kSolveRhs * esz);
  const size_t o_W = cv.take<char>((size_t)ldy * kSolveRhs * esz);
  const size_t o_box = cv.take<uint64_t>((size_t)nblk * kSolveRhs * 64 * 2);
  const size_t o_dinv = cv.take<char>((size_t)(1 + 2 * 2) * nblk * 64 * 64 * esz);
  void* ws = nullptr;
  int* status = nullptr;
  hipError_t e = workspace(cv.off, stream, &ws, &status);
  if (e != hipSuccess) return hip_err(e);
  char* base = static_cast<char*>(ws);
  SolveWork w{};
  w.perm = reinterpret_cast<int*>(base + o_perm);
  w.cnt = reinterpret_cast<int*>(base + o_cnt);
  w.off = reinterpret_cast<int*>(base + o_off);
  w.list = reinterpret_cast<int*>(base + o_list);
  w.alpha = base + o_al;
  w.ralpha = base + o_ral;
  w.Y = base + o_Y;
  w.W = base + o_W;
  w.ldy = ldy;
  w.box = reinterpret_cast<uint64_t*>(base + o_box);
  w.dinv = base + o_dinv;
  w.status = status;
  e = launch_init(nullptr, 0, status, stream);    // clear the bounded-wait flag
  if (e == hipSuccess) {
    if (dtype == LTLT_F64)
      e = launch_solve<double>((int)n, static_cast<const double*>(A), lda, ipiv, (int)nrhs, static_cast<double*>(B),
                               ldb, w, stream);
    else
      e = launch_solve<float>((int)n, static_cast<const float*>(A), lda, ipiv, (int)nrhs, static_cast<float*>(B),
                              ldb, w, stream);
  }
  return e == hipSuccess ? 0 : hip_err(e);
}

int ltlt_factor_batched(int64_t n, int64_t batch, void* A, int64_t lda, int64_t strideA, int dtype,
                        int32_t* ipiv, int64_t strideIpiv, double* logabs, int32_t* sign, hipStream_t stream) {
  if (n < 0 || n > LTLT_BATCHED_MAX_N) return -1;
  if (batch < 0 || batch > (int64_t)INT32_MAX) return -2;
  if (A == nullptr && n > 0 && batch > 0) return -3;
  if (lda < std::max<int64_t>(1, n)) return -4;
  if (batch > 1 && strideA < lda * n) return -5;
  if (bad_dtype(dtype)) return -6;
  if (ipiv == nullptr && n > 0 && batch > 0) return -7;
  if (batch > 1 && strideIpiv < n) return -8;
  if (logabs == nullptr && batch > 0) return -9;
  if (sign == nullptr && batch > 0) return -10;
  if (batch == 0) return 0;
  hipError_t e;
  if (dtype == LTLT_F64)
    e = launch_batched<double>((int)n, (int)batch, static_cast<double*>(A), lda, strideA, ipiv, strideIpiv, logabs,
                               sign, stream);
  else
    e = launch_batched<float>((int)n, (int)batch, static_cast<float*>(A), lda, strideA, ipiv, strideIpiv, logabs,
                              sign, stream);
  return e == hipSuccess ? 0 : hip_err(e);
}

int ltlt_skew_update(int64_t m, void* C, int64_t ldc, const int32_t* perm, int64_t K, const void* Lx, int64_t ldl,
                     const void* Bt, int64_t ldb, int dtype, hipStream_t stream) {
  if (m < 0 || m > (int64_t)INT32_MAX / 2) return -1;
  if (C == nullptr && m > 0) return -2;
  if (ldc < std::max<int64_t>(1, m)) return -3;
  if (K < 0 || K > (int64_t)INT32_MAX / 2) return -5;
  if (Lx == nullptr && m > 0 && K > 0) return -6;
  if (ldl < std::max<int64_t>(1, m)) return -7;
  if (Bt == nullptr && m > 0 && K > 0) return -8;
  if (ldb < std::max<int64_t>(1, m)) return -9;
  if (bad_dtype(dtype)) return -10;
  if (m < 2) return 0;
  UpdateArgs ua{};
  ua.C = C; ua.ldc = ldc; ua.m = (int)m; ua.perm = perm; ua.perm_base = 0;
  ua.perm_lo = INT32_MIN; ua.perm_hi = INT32_MAX;   // the caller's sources, as given
  ua.K = (int)K; ua.Lx = Lx; ua.ldl = ldl; ua.Bt = Bt; ua.ldb = ldb;
  hipError_t e = dtype == LTLT_F64 ? launch_update<double>(ua, stream) : launch_update<float>(ua, stream);
  return e == hipSuccess ? 0 : hip_err(e);
}

int ltlt_device_status(hipStream_t stream) {
  hipError_t e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_err(e);
  int dev = 0;
  e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_err(e);
  int* st = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (dev < 0 || dev >= kMaxScratchDevices || !g_scratch_ptr[dev]) return 0;   // no call on this device yet
    st = reinterpret_cast<int*>(g_scratch_ptr[dev]);
  }
  // the sticky word: raised by any wait that gave up since the last read
  int h = 0;
  e = hipMemcpy(&h, st + 1, sizeof(int), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_err(e);
  if (h != 0) {
    e = hipMemset(st + 1, 0, sizeof(int));
    if (e != hipSuccess) return hip_err(e);
    return LTLT_ERR_DEVICE_TIMEOUT;
  }
  return 0;
}

int ltlt_test_force_timeout(int on) {
  if (on != 0 && on != 1) return -1;
  ltlt::g_forced_timeout.store(on == 1, std::memory_order_relaxed);
  return 0;
}

int ltlt_profile_enable(int on) {
  if (on < 0 || on > 2) return -1;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (on) prof_clear_locked();
  g_prof_on = on != 0;
  g_prof_update_only = on == 2;
  return 0;
}

int ltlt_profile_read(int nkinds, int64_t* launches, double* ms, double* flops) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  const int kinds = std::min(nkinds, 4);
  for (int k = 0; k < kinds; ++k) { launches[k] = 0; ms[k] = 0.0; flops[k] = 0.0; }
  for (auto& r : g_prof) {
    hipError_t e = hipEventSynchronize(r.b);
    if (e != hipSuccess) return hip_err(e);
    float t = 0.f;
    e = hipEventElapsedTime(&t, r.a, r.b);
    if (e != hipSuccess) return hip_err(e);
    if (r.kind < kinds) {
      launches[r.kind] += 1;
      ms[r.kind] += t;
      flops[r.kind] += r.flops;
    }
  }
  return kinds;
}

int ltlt_set_cooperative_panels(int on) {
  if (on != 0 && on != 1) return -1;
  ltlt::g_cooperative_panels.store(on == 1, std::memory_order_relaxed);
  return 0;
}

int ltlt_release_workspace(void) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  int dev0 = 0;
  (void)hipGetDevice(&dev0);
  for (auto& kv : g_ws) {
    if (hipSetDevice(kv.first) != hipSuccess) continue;
    (void)hipDeviceSynchronize();
    if (kv.second.ptr) (void)hipFree(kv.second.ptr);
  }
  g_ws.clear();
  (void)hipSetDevice(dev0);
  return 0;
}

}  // extern "C"
