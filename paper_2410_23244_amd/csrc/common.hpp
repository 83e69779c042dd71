// common.hpp -- layouts shared by the host library and the kernels of libbart.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bart.h"

namespace bart {

constexpr int kBlock = 512;           // threads per workgroup of the sweep kernel (256 VGPRs each)
constexpr int kWaves = kBlock / 64;   // wave64 on CDNA4
constexpr int kMaxLeaves = 128;       // leaves of a depth-8 heap tree
constexpr int kStride = 144;          // 64-bit words per mailbox (>= kMaxLeaves + 1, 128-byte lines)
constexpr int kBinFloats = 32768;     // 128 KiB of LDS per-leaf bins
constexpr int kMaxGrid = 256;         // mailboxes per buffer reserved in the workspace
constexpr int kMaxLaunchSteps = (1 << 20) - 8;  // steps per launch (20-bit sequence numbers)

enum Move : int32_t { kNone = 0, kGrow = 1, kPrune = 2 };

// Global-address-space view of a device pointer.  Pointers read out of the
// argument block are generic ("flat") to the compiler; flat loads count
// against the LDS wait counter too, so an LDS read would stall behind every
// outstanding HBM load.  Kernels access device memory through gbl(p).
template <class T>
using gptr = __attribute__((address_space(1))) T *;
template <class T>
__device__ __forceinline__ gptr<T> gbl(T *p) {
  return (gptr<T>)p;
}

// Proposal of one tree for its step of the current sweep (sec. 3.3 items 1
// and 6: everything that does not depend on residuals), 96 bytes.
struct Prop {
  int32_t move, eta, axis, cut;
  int32_t nG, nP, L, rank_l;  // #G(T), #P(T), leaves of the larger tree, rank of 2*eta
  int32_t rank_r, pad0, pad1, pad2;
  uint64_t mask[4];           // bit h set iff heap slot h is a leaf of the larger tree
  double c_prior;             // log r minus the marginal-likelihood term
  double ln_u;                // log of the accept uniform
};
static_assert(sizeof(Prop) == 96, "Prop layout");

// Scalars the kernels keep in device memory.
struct Ctl {
  double sigma2;
  int64_t sweep;
  uint32_t error;
  uint32_t pad;
  uint64_t stats[6];  // GROW proposed, PRUNE proposed, GROW accepted, PRUNE accepted, tree steps, leaves
};

// Arguments of one chain.  A launch covers nchain chains with G workgroups
// each; workgroup b serves chain b / G, whose arguments are entry b / G of
// the array the kernel receives.  Per-chain buffers are disjoint; X, n_cuts,
// nz_list and nz_rank are shared.
struct SweepArgs {
  const uint8_t *X;
  int64_t ldx;
  float *resid;
  void *idx;
  int64_t ldi;  // entries between index-cache rows
  uint16_t *axis;
  uint8_t *cut;
  float *leaf;
  int32_t *count;
  Prop *prop;
  double *z;  // [2][m][2H] leaf normals, by sweep parity
  const int32_t *n_cuts;
  const int32_t *nz_list;
  const int32_t *nz_rank;
  Ctl *ctl;
  uint64_t *pub;     // [2][G][kStride] mailboxes, by step parity
  int32_t n, p, m, D, H, p_nz, G, chunks;
  int32_t cpt;    // chunks of 4 observations per thread
  int32_t chain;  // index of this chain in the launch
  float *latent;        // probit: [n_pad] latents of this chain
  const uint8_t *ybin;  // probit: [n_pad] binary response (shared)
  int32_t probit, pad2_;
  double probit_offset;
  double alpha, beta, mu_mu, sigma_mu, nu, lambda, p_grow;
};

// What changes from one launch of the sweep kernel to the next.
struct Launch {
  int64_t s0;         // sweep of the first step
  int32_t j0;         // first step inside that sweep (0..m-1 trees, m = sigma^2)
  int32_t n_steps;
  uint64_t seed;
  bart_trace *trace;  // NULL: no trace; else [nchain][trace_stride] records
  int64_t trace_stride;
  uint32_t spin_limit;  // poll rounds before a cross-workgroup wait gives up
  int32_t absent_wg;    // -1; else a workgroup that returns at once (the timeout test)
};

// Index of the calling workgroup among the G workgroups of its chain.
__device__ __forceinline__ int wg_id(const SweepArgs *__restrict__ A) {
  return (int)blockIdx.x - A->chain * A->G;
}

}  // namespace bart
