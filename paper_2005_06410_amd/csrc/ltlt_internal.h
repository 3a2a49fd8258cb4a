// Internal declarations shared by the host driver and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ltlt {

constexpr int kThreads = 256;        // workgroup size of the update kernel
constexpr int kMaxNb = 256;          // widest panel
constexpr int kPanelThreads = 512;          // workgroup size of the panel kernel
constexpr int kPanelWaves = kPanelThreads / 64;   // waves per panel workgroup
constexpr int kMaxPanelRecords = 256;       // exchange records one poll covers (4 per lane)
constexpr int kRecStride = 32;              // 64-bit words from one exchange record to the next (256 bytes)

// Arguments of one panel launch (block of steps k = j .. j+bw-1).
struct PanelArgs {
  const void* A;      // matrix, column-major, strict lower triangle as of block start
  int64_t lda;
  int n;
  int j;              // first column step of the block
  int bw;             // steps in the block
  int R;              // rows per workgroup
  int P;              // workgroups
  int nrec;           // exchange records per slot (>= P of every block)
  void* G;            // multipliers by block-start index: G[(idx - j - 1) + u*ldw]
  void* PO;           // panel out, rows j+1.., columns 0..bw (bw = carry), ld = ldw
  void* Bm;           // Bt = Lx Tx^T for rows >= j+bw+1, columns 0..bw, ld = ldw
  int64_t ldw;
  void* alpha;        // alpha_{j+t}, t < bw
  int* perm;          // perm[i] for positions i >= j+1: index held at block start
  int* ipiv;
  uint64_t* rec;      // exchange records [2][nrec][kRecStride] (words 0, 1 used)
  int* status;        // nonzero: a bounded wait gave up
};

// Arguments of one trailing update.
struct UpdateArgs {
  void* C;            // first element of the m x m trailing block
  int64_t ldc;
  int m;
  const int* perm;    // source index per row/column (minus perm_base), or nullptr
  int perm_base;
  int perm_lo, perm_hi;   // relative sources are clamped into [perm_lo, perm_hi]
  int K;
  const void* Lx;
  int64_t ldl;
  const void* Bt;
  int64_t ldb;
  int pad_row;        // nonzero: row m of every Lx / Bt column is readable (workspace padding)
  int tiles;          // number of 128-row tile rows
};

// Launch of a grid whose workgroups wait on each other every step (the
// panels: at most one workgroup per CU, never more workgroups than the
// device holds at once).  By default an ordinary launch: issued in stream
// order onto an otherwise idle device, every workgroup is dispatched at
// once, and every wait is bounded, so a grid that cannot become resident
// (other streams or processes holding CUs for seconds) fails with the
// bounded-wait status instead of hanging.  ltlt_set_cooperative_panels(1)
// selects the runtime's cooperative launch, which guarantees co-residency
// at a cost of about 20 us per launch.
bool cooperative_panels();
template <typename K, typename A>
hipError_t launch_resident_grid(K kernel, unsigned grid, unsigned block, size_t lds, hipStream_t s, const A& arg) {
  A copy = arg;
  void* args[] = {&copy};
  if (cooperative_panels())
    return hipLaunchCooperativeKernel((const void*)kernel, dim3(grid), dim3(block), args, (unsigned)lds, s);
  return hipLaunchKernel((const void*)kernel, dim3(grid), dim3(block), args, lds, s);
}

template <typename T> hipError_t launch_panel(const PanelArgs& a, size_t lds, hipStream_t s);
template <typename T> size_t panel_lds_bytes(int bw, int R);
template <typename T> hipError_t launch_update(const UpdateArgs& a, hipStream_t s);

template <typename T> hipError_t launch_commit(T* A, int64_t lda, int n, int j, int bw, const T* PO,
                                               int64_t ldw, const T* alpha, const int* status, hipStream_t s);
template <typename T> hipError_t launch_perm_apply(T* A, int64_t lda, int n, const int* G, int nb, int c_end,
                                                   T* stage, hipStream_t s);
template <typename T> size_t perm_stage_elems(int n, int c_end);
template <typename T> hipError_t launch_pfaffian(int n, const T* A, int64_t lda, const int* ipiv, double* logabs,
                                                 int* sign, const int* status, hipStream_t s);
template <typename T> hipError_t launch_batched(int n, int batch, T* A, int64_t lda, int64_t strideA, int* ipiv,
                                                int64_t strideIpiv, double* logabs, int* sign, hipStream_t s);

hipError_t launch_init(int* ipiv, int n, int* status, hipStream_t s);
// Host-side switch for the failure-path test: while set, every call's init
// raises the status words as if a wait had given up (ltlt_test_force_timeout).
bool forced_timeout();
// Raises a kernel's dynamic-LDS limit to `bytes` on the current device, once
// per (kernel, device): the attribute is per device.  Thread-safe.
hipError_t ensure_dynamic_lds(const void* kernel, int bytes);
hipError_t launch_rec_init(uint64_t* rec, int nrec_per_slot, hipStream_t s);
hipError_t launch_perm_chain(const int* Tblk, int nb, int nblk, int n, int* G, hipStream_t s);
template <typename T> int panel_max_blocks(int bw, size_t lds);
int panel_rows(int bw);

// Complex matrices are factored as two real planes (real and imaginary parts,
// leading dimension ldw).  The complex panel writes its outputs so that each
// plane's trailing update is one real product of depth 2K (K = bw + 1):
//   Re C += [Lr Li] [Btr -Bti]^T,   Im C += [Li Lr] [Btr Bti]^T,
// with LL = [Lr Li Lr] holding both left operands as column windows.
struct CPanelArgs {
  PanelArgs b;        // A, G, alpha: real planes / parts; PO and Bm unused
  const void* Ai;     // imaginary plane of the matrix (ld b.lda)
  void* Gi;           // imaginary plane of the multiplier copy G
  void* Vr;           // pivot candidates' values by block-start index:
  void* Vi;           //   V[idx - j - 1] (real and imaginary parts)
  void* LL;           // [Lr | Li | Lr], K columns each, ld b.ldw, rows from j+1
  void* BtA;          // [Btr | -Bti] for rows >= j+bw+1, ld b.ldw
  void* BtB;          // [Btr |  Bti]
  void* alpha_i;      // imaginary parts of alpha_{j+t}
};
int cpanel_rows(int bw);
template <typename T> size_t cpanel_lds_bytes(int bw);
template <typename T> int cpanel_max_blocks(int bw, size_t lds);
template <typename T> hipError_t launch_cpanel(const CPanelArgs& a, size_t lds, hipStream_t s);
template <typename T> hipError_t launch_cplx_split(int n, const void* A, int64_t lda, T* Pr, T* Pi, int64_t ldp,
                                                   hipStream_t s);
template <typename T> hipError_t launch_cplx_merge(int n, void* A, int64_t lda, const T* Pr, const T* Pi,
                                                   int64_t ldp, hipStream_t s);
template <typename T> hipError_t launch_cpfaffian(int n, const void* A, int64_t lda, const int* ipiv,
                                                  double* logabs, double* phase, const int* status, hipStream_t s);

// Solve with the factors.
constexpr int kSolveRhs = 8;                    // right-hand sides per pass
struct SolveWork {
  int* perm;          // [n]
  int* cnt;           // [2n] counters (steps per target position, fill)
  int* off;           // [n+1] bucket offsets
  int* list;          // [n] steps by target position
  void* alpha;        // [n] alpha_k
  void* ralpha;       // [n] 1 / alpha_k
  void* Y;            // [ldy][kSolveRhs]
  void* W;            // [ldy][kSolveRhs]
  int64_t ldy;
  uint64_t* box;      // [blocks][kSolveRhs][64][2] stamped solution words
  int* status;
  void* dinv;         // [1 + 2 * 2][blocks][64 * 64]: inverses of the diagonal blocks of L and
                      // the matrices of the last two dependencies of each substitution
};
template <typename T> hipError_t launch_solve(int n, const T* A, int64_t lda, const int* ipiv, int nrhs, T* B,
                                              int64_t ldb, const SolveWork& w, hipStream_t s);

// Pfaffian-only path (even column steps): the pair panel and the commit of
// its alphas.
int pair_panel_rows(int bw);                     // rows per pair-panel workgroup
template <typename T> size_t pair_lds_bytes(int bw, int R);
template <typename T> int pair_max_blocks(int bw, size_t lds);
template <typename T> hipError_t launch_pair_panel(const PanelArgs& a, size_t lds, hipStream_t s);
template <typename T> hipError_t launch_pair_commit(T* A, int64_t lda, int j, int nt, const T* alpha,
                                                    const int* status, hipStream_t s);

}  // namespace ltlt
