// bart.hip -- host side of libbart: validation, workspace carving, launches.
// The C ABI is declared and documented in include/bart.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"
#include "sweep.hpp"

using namespace bart;

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                              \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess)                                                          \
      return fail(BART_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_));       \
  } while (0)

constexpr size_t kAlign = 256;
size_t up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Workspace: nchain chain blocks of chain_bytes each (offsets resid..pub are
// relative to a block), then the shared part (offsets n_cuts..args absolute).
struct Layout {
  int64_t n_pad;
  int32_t nchain;
  int32_t gcap;  // workgroups per chain the mailboxes are sized for
  size_t resid, idx, axis, cut, leaf, count, prop, z, ctl, pub, latent, chain_bytes;
  size_t n_cuts, nz_list, nz_rank, ybin, args, args_static, total;
};

int nchain_of(const bart_config &c) { return c.nchain > 0 ? c.nchain : 1; }

const char *check_config(const bart_config *c) {
  if (!c) return "config is NULL";
  if (c->n < 1) return "n must be >= 1";
  if (c->p < 1 || c->p > 65535) return "p must be in [1, 65535]";
  if (c->ntree < 1) return "ntree must be >= 1";
  if (c->max_depth < 2 || c->max_depth > 8) return "max_depth must be in [2, 8]";
  if (c->idx_bytes < 0 || c->idx_bytes > 2) return "idx_bytes must be 0, 1 or 2";
  if (c->idx_bytes == 0 && c->residency == BART_RESID_REGISTERS)
    return "idx_bytes = 0 (no index cache) needs streamed residuals";
  if (c->grid < 0 || c->grid > kMaxGrid) return "grid must be 0 or in [1, 256]";
  if (c->nchain < 0 || c->nchain > kMaxGrid) return "nchain must be 0 or in [1, 256]";
  if (c->grid > 0 && (int64_t)c->grid * nchain_of(*c) > kMaxGrid)
    return "grid x nchain must not exceed 256";
  if (c->launch != BART_LAUNCH_COOPERATIVE && c->launch != BART_LAUNCH_ORDINARY)
    return "launch must be BART_LAUNCH_COOPERATIVE or BART_LAUNCH_ORDINARY";
  if (c->residency < BART_RESID_AUTO || c->residency > BART_RESID_STREAMED)
    return "residency must be BART_RESID_AUTO, BART_RESID_REGISTERS or BART_RESID_STREAMED";
  if (c->x_stride < c->n || c->x_stride % 16) return "x_stride must be >= n and a multiple of 16";
  if (!(c->alpha >= 0.0 && c->alpha <= 1.0)) return "alpha must be in [0, 1]";
  if (!(c->beta >= 0.0 && std::isfinite(c->beta))) return "beta must be finite and >= 0";
  if (!std::isfinite(c->mu_mu)) return "mu_mu must be finite";
  if (!(c->sigma_mu > 0.0 && std::isfinite(c->sigma_mu))) return "sigma_mu must be > 0";
  if (!(c->nu > 0.0 && std::isfinite(c->nu))) return "nu must be > 0";
  if (!(c->lambda > 0.0 && std::isfinite(c->lambda))) return "lambda must be > 0";
  if (!(c->sigma2_init > 0.0 && std::isfinite(c->sigma2_init))) return "sigma2_init must be > 0";
  if (!(c->p_grow >= 0.0 && c->p_grow <= 1.0)) return "p_grow must be in [0, 1]";
  if (c->nu + (double)c->n < 2.0) return "nu + n must be >= 2 (gamma shape >= 1)";
  if (c->probit != 0 && c->probit != 1) return "probit must be 0 or 1";
  if (c->probit && !std::isfinite(c->probit_offset)) return "probit_offset must be finite";
  return nullptr;
}

Layout make_layout(const bart_config &c) {
  Layout L{};
  const int64_t H = 1 << (c.max_depth - 1);
  const int64_t m = c.ntree;
  L.n_pad = (int64_t)up((size_t)c.n, 256);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = up(o + bytes, kAlign);
    return at;
  };
  L.nchain = nchain_of(c);
  L.gcap = kMaxGrid / L.nchain;
  L.resid = take(sizeof(float) * L.n_pad);
  // without an index cache: two rolling rows of u8 leaf indices
  L.idx = take(c.idx_bytes ? (size_t)m * L.n_pad * c.idx_bytes : 2 * (size_t)L.n_pad);
  L.axis = take(sizeof(uint16_t) * m * H);
  L.cut = take(m * H);
  L.leaf = take(sizeof(float) * m * 2 * H);
  L.count = take(sizeof(int32_t) * m * 2 * H);
  L.prop = take(sizeof(Prop) * m);
  L.z = take(sizeof(double) * 2 * m * 2 * H);
  L.ctl = take(sizeof(Ctl));
  L.pub = take(sizeof(uint64_t) * 2 * L.gcap * kStride);
  L.latent = take(c.probit ? sizeof(float) * L.n_pad : 0);
  L.chain_bytes = o;
  o = L.chain_bytes * L.nchain;
  L.n_cuts = take(sizeof(int32_t) * c.p);
  L.nz_list = take(sizeof(int32_t) * c.p);
  L.nz_rank = take(sizeof(int32_t) * c.p);
  L.ybin = take(c.probit ? L.n_pad : 0);
  L.args = take(sizeof(SweepArgs) * L.nchain);
  // the same arguments with the mailboxes in the library's static scratch
  // array (bart_step_static)
  L.args_static = take(sizeof(SweepArgs) * L.nchain);
  L.total = o;
  return L;
}

using SweepFn = void (*)(const SweepArgs *, Launch);
constexpr int kVs[] = {1, 2, 4, 8};

template <int IB>
SweepFn regs_fn(int V) {
  switch (V) {
    case 1: return sweep_kernel<1, IB>;
    case 2: return sweep_kernel<2, IB>;
    case 4: return sweep_kernel<4, IB>;
    case 8: return sweep_kernel<8, IB>;
  }
  return nullptr;
}

SweepFn sweep_fn(int V, int IB) { return IB == 1 ? regs_fn<1>(V) : regs_fn<2>(V); }

// IB = 0: no index cache (Algorithm 1 per tree step); the rank stash when a
// thread's chunks fit it
template <bool ST>
SweepFn stream_fn_st(int IB) {
  return IB == 0 ? sweep_kernel_stream<1, true, ST>
                 : (IB == 1 ? sweep_kernel_stream<1, false, ST> : sweep_kernel_stream<2, false, ST>);
}
SweepFn stream_fn(int IB, int cpt) {
  return cpt <= kStashCpt ? stream_fn_st<true>(IB) : stream_fn_st<false>(IB);
}

// ------------------------------------------------------- static scratch
// Mailboxes of bart_step_static: a file-scope device array instead of the
// workspace, for callers that cannot allocate.  Chain c of a handle with
// nchain chains uses words [c, c + 1) x kStaticChainWords with
// kStaticChainWords = 2 (kMaxGrid / nchain) kStride: the same per-chain
// capacity the workspace reserves.  Each device holds its own copy; host
// code never uses the array's name as an address, only the per-device
// address from hipGetSymbolAddress (scratch_ptr).
constexpr int64_t kScratchWords = 2 * (int64_t)kMaxGrid * kStride;  // 576 KiB
static __device__ __align__(256) uint64_t scratch[kScratchWords];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint64_t *g_scratch[kMaxDevices];  // device address of scratch, per device

// The address of this device's scratch array; looked up once per device,
// with that device current (bart_init).
int scratch_ptr(int device, uint64_t **out) {
  if (device < 0 || device >= kMaxDevices)
    return fail(BART_ENOTSUP, "device %d beyond the %d devices the library tracks", device,
                kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[device]) {
    void *p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(BART_EHIP, "hipGetSymbolAddress returned NULL for the scratch array");
    g_scratch[device] = (uint64_t *)p;
  }
  *out = g_scratch[device];
  return BART_OK;
}

// ---------------------------------------------------------------- kernels

__global__ void k_init_resid(float *resid, const float *y, int64_t n, int64_t n_pad) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n_pad;
       i += (int64_t)gridDim.x * blockDim.x)
    resid[i] = i < n ? y[i] : 0.f;
}

// Probit start: y_i = [y_c[i] > 0], latent z_i = +-1 on its side of 0,
// residual z_i - offset (every tree is zero); padding gets y = 0, z = r = 0.
__global__ void k_init_probit(const float *y, uint8_t *ybin, float *latent, float *resid,
                              double offset, int64_t n, int64_t n_pad) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n_pad;
       i += (int64_t)gridDim.x * blockDim.x) {
    const bool valid = i < n;
    const int yb = valid && y[i] > 0.f;
    const float z = valid ? (yb ? 1.f : -1.f) : 0.f;
    if (ybin) ybin[i] = (uint8_t)yb;
    latent[i] = z;
    resid[i] = valid ? (float)((double)z - offset) : 0.f;
  }
}

// Every observation starts in the root (slot 1); padding entries of a row
// (n <= i < n_pad) hold 0, a slot that is never a leaf.
__global__ void k_fill_idx(uint8_t *idx, int64_t entries, int ib, int64_t n, int64_t n_pad) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < entries;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int v = i % n_pad < n ? 1 : 0;
    if (ib == 1)
      idx[i] = (uint8_t)v;
    else
      ((uint16_t *)idx)[i] = (uint16_t)v;
  }
}

// Padding entries (n <= i < n_pad) of m index rows back to 0.
__global__ void k_zero_idx_pad(uint8_t *idx, int ib, int64_t n, int64_t n_pad, int64_t m) {
  const int64_t per = n_pad - n;
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < m * per;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = (q / per) * n_pad + n + q % per;
    if (ib == 1)
      idx[i] = 0;
    else
      ((uint16_t *)idx)[i] = 0;
  }
}

__global__ void k_init_trees(uint16_t *axis, uint8_t *cut, float *leaf, int32_t *count, int64_t m,
                             int H, int32_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < m * 2 * H;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int h = (int)(i % (2 * H));
    leaf[i] = 0.f;
    count[i] = h == 1 ? n : 0;
    if (h < H) {
      const int64_t q = (i / (2 * H)) * H + h;
      axis[q] = 0;
      cut[q] = 0;
    }
  }
}

// sigma2 < 0 keeps the current value
__global__ void k_set_ctl(Ctl *ctl, double sigma2, int64_t sweep, int reset_stats) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    if (sigma2 >= 0.0) ctl->sigma2 = sigma2;
    ctl->sweep = sweep;
    if (reset_stats) {
      ctl->error = 0;
      for (int k = 0; k < 6; ++k) ctl->stats[k] = 0;
    }
  }
}

__global__ void k_clear_words(uint64_t *p, int64_t words) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < words;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

// The mailboxes of every chain: words at byte offset off of each chain block
// (blockIdx.y = chain).
__global__ void k_clear_mailboxes(char *ws, size_t off, size_t chain_bytes, int64_t words) {
  uint64_t *p = (uint64_t *)(ws + blockIdx.y * chain_bytes + off);
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < words;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

__global__ void k_zero_i32(int32_t *p, int64_t count) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

// Leaf of every observation in every tree (blockIdx.y) by Algorithm 1: into
// out [m][n] u8 and/or as per-leaf counts (an LDS histogram per block).
__global__ void k_leaf_index(const uint8_t *X, int64_t ldx, int64_t n, int p, const uint16_t *axis,
                             const uint8_t *cut, int D, int H, uint8_t *out, int32_t *count) {
  __shared__ int hist[256];
  const int j = blockIdx.y;
  for (int k = threadIdx.x; k < 256; k += blockDim.x) hist[k] = 0;
  __syncthreads();
  const uint16_t *ax = axis + (int64_t)j * H;
  const uint8_t *ct = cut + (int64_t)j * H;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    int h = 1;
    for (int lvl = 1; lvl < D; ++lvl) {
      const int cv = ct[h];
      if (cv == 0) break;
      const int a = ax[h] < p ? ax[h] : 0;
      h = 2 * h + (X[(int64_t)a * ldx + i] >= cv ? 1 : 0);
      if (h >= H) break;
    }
    if (out) out[(int64_t)j * n + i] = (uint8_t)h;
    if (count) atomicAdd(&hist[h], 1);
  }
  __syncthreads();
  if (count)
    for (int k = threadIdx.x; k < 2 * H; k += blockDim.x)
      if (hist[k]) atomicAdd(&count[(int64_t)j * 2 * H + k], hist[k]);
}

// Per-leaf counts of every tree from the index cache (after a state load).
// Leaf counts of every tree from the index cache; an entry of a real
// observation outside slots 1..2H-1 (0 marks padding) flags the cache as
// inconsistent.
__global__ void k_recount(const uint8_t *idx, int64_t ldi, int ib, int32_t *count, int32_t n,
                          int H, uint32_t *error) {
  __shared__ int hist[256];
  const int j = blockIdx.y;
  for (int k = threadIdx.x; k < 256; k += blockDim.x) hist[k] = 0;
  __syncthreads();
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int v = ib == 1 ? idx[j * ldi + i] : ((const uint16_t *)idx)[j * ldi + i];
    if (v >= 1 && v < 2 * H)
      atomicAdd(&hist[v], 1);
    else
      atomicOr(error, BART_DEVERR_CACHE);
  }
  __syncthreads();
  for (int k = threadIdx.x; k < 2 * H; k += blockDim.x)
    if (hist[k]) atomicAdd(&count[(int64_t)j * 2 * H + k], hist[k]);
}

// f(x) = offset + sum_j g(x; T_j, M_j): Algorithm 1 per tree (loop over the
// levels with a reached-leaf flag), fp64 sum in tree order.  Trees are staged
// through LDS in tiles of kPredNodes heap slots; every thread follows its
// point through kPredIlp trees at once so their predictor-byte gathers
// overlap.  blockIdx.y = chain: its trees sit chain_bytes further on, its
// outputs nt further on.  ACC: add f and f^2 (fp64) to sum and sumsq instead
// of writing fp32(f) to out.
constexpr int kPredBlock = 256;
constexpr int kPredNodes = 2048;  // heap slots per LDS tile (axis u16 + cut u8 + 2 leaves f32: 22 KB)
constexpr int kPredIlp = 8;

template <bool ACC>
__global__ void __launch_bounds__(kPredBlock)
    k_predict(const uint8_t *Xt, int64_t ldx, int64_t nt, int p, const uint16_t *axis0,
              const uint8_t *cut0, const float *leaf0, int m, int D, int H, double offset,
              size_t chain_bytes, float *out0, double *sum0, double *sumsq0) {
  __shared__ uint16_t s_ax[kPredNodes];
  __shared__ uint8_t s_ct[kPredNodes];
  __shared__ float s_lf[2 * kPredNodes];
  const int t = threadIdx.x;
  const int64_t i = blockIdx.x * (int64_t)kPredBlock + t;
  const bool valid = i < nt;
  const size_t cb = blockIdx.y * chain_bytes;
  const uint16_t *axis = (const uint16_t *)((const char *)axis0 + cb);
  const uint8_t *cut = cut0 + cb;
  const float *leaf = (const float *)((const char *)leaf0 + cb);
  const int TT = kPredNodes / H;  // trees per tile
  const uint8_t *xcol = Xt + (valid ? i : 0);
  double acc = 0.0;
  for (int j0 = 0; j0 < m; j0 += TT) {
    const int nt_ = min(TT, m - j0);
    __syncthreads();
    for (int q = t; q < nt_ * H; q += kPredBlock) {
      s_ax[q] = axis[(int64_t)j0 * H + q];
      s_ct[q] = cut[(int64_t)j0 * H + q];
    }
    for (int q = t; q < nt_ * 2 * H; q += kPredBlock) s_lf[q] = leaf[(int64_t)j0 * 2 * H + q];
    __syncthreads();
    if (!valid) continue;
    for (int jj = 0; jj < nt_; jj += kPredIlp) {
      int index[kPredIlp];
      bool found[kPredIlp];
#pragma unroll
      for (int u = 0; u < kPredIlp; ++u) {
        index[u] = 1;
        found[u] = jj + u >= nt_;  // past the tile: nothing to do
      }
      for (int lvl = 1; lvl <= D - 1; ++lvl) {
#pragma unroll
        for (int u = 0; u < kPredIlp; ++u) {
          const int base = (jj + u < nt_ ? jj + u : 0) * H;
          const int a = s_ax[base + index[u]], split = s_ct[base + index[u]];
          found[u] = found[u] || split == 0;
          const int xa = found[u] ? 0 : xcol[(int64_t)(a < p ? a : 0) * ldx];
          index[u] = found[u] ? index[u] : 2 * index[u] + (xa >= split ? 1 : 0);
        }
      }
#pragma unroll
      for (int u = 0; u < kPredIlp; ++u)  // tree order
        if (jj + u < nt_) acc += (double)s_lf[(jj + u) * 2 * H + index[u]];
    }
  }
  if (!valid) return;
  const int64_t o = blockIdx.y * nt + i;
  const double f = offset + acc;
  if (ACC) {
    sum0[o] += f;
    sumsq0[o] += f * f;
  } else {
    out0[o] = (float)f;
  }
}

// Posterior mean and sd of f at each point from the per-chain sums of f and
// f^2 over n_keep kept sweeps: chain means m_c and variances v_c = E_c[f^2] -
// m_c^2, pooled by the law of total variance (mean of the v_c plus the
// variance of the m_c over the chains); one thread per point, fp64.
__global__ void k_posterior_summary(const double *sum, const double *sumsq, int64_t nt, int nchain,
                                    double inv_keep, double *mean, double *sd) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nt;
       i += (int64_t)gridDim.x * blockDim.x) {
    double mbar = 0.0;
    for (int c = 0; c < nchain; ++c) mbar += sum[c * nt + i] * inv_keep;
    mbar /= nchain;
    double within = 0.0, between = 0.0;
    for (int c = 0; c < nchain; ++c) {
      const double mc = sum[c * nt + i] * inv_keep;
      within += sumsq[c * nt + i] * inv_keep - mc * mc;
      between += (mc - mbar) * (mc - mbar);
    }
    const double var = (within + between) / nchain;
    mean[i] = mbar;
    sd[i] = var > 0.0 ? sqrt(var) : 0.0;
  }
}

int grid_for(int64_t work, int block) {
  int64_t g = (work + block - 1) / block;
  return (int)std::max<int64_t>(1, std::min<int64_t>(g, 65536));
}

}  // namespace

struct bart_handle {
  bart_config cfg;
  Layout lay;
  char *ws;
  const uint8_t *X;
  hipStream_t stream;
  int device;
  int H, p_nz, V, G, lds;  // V: chunks of 4 observations per thread; G: workgroups per chain
  int nchain;
  bool streamed;           // residuals streamed from HBM instead of kept in registers
  int64_t chunks;
  int64_t sweep;
  int32_t next;
  std::vector<int32_t> n_cuts, nz_list, nz_rank;
  SweepFn fn;
  uint64_t *scratch_dev;  // device address of this device's scratch array
};

namespace {

// shared part of the workspace
template <class T>
T *at(bart_handle *h, size_t off) {
  return (T *)(h->ws + off);
}

// block of chain c
template <class T>
T *atc(bart_handle *h, int c, size_t off) {
  return (T *)(h->ws + (size_t)c * h->lay.chain_bytes + off);
}

SweepArgs make_args(bart_handle *h, int ch) {
  const bart_config &c = h->cfg;
  SweepArgs A{};
  A.X = h->X;
  A.ldx = c.x_stride;
  A.resid = atc<float>(h, ch, h->lay.resid);
  A.idx = atc<void>(h, ch, h->lay.idx);
  A.ldi = h->lay.n_pad;
  A.axis = atc<uint16_t>(h, ch, h->lay.axis);
  A.cut = atc<uint8_t>(h, ch, h->lay.cut);
  A.leaf = atc<float>(h, ch, h->lay.leaf);
  A.count = atc<int32_t>(h, ch, h->lay.count);
  A.prop = atc<Prop>(h, ch, h->lay.prop);
  A.z = atc<double>(h, ch, h->lay.z);
  A.n_cuts = at<int32_t>(h, h->lay.n_cuts);
  A.nz_list = at<int32_t>(h, h->lay.nz_list);
  A.nz_rank = at<int32_t>(h, h->lay.nz_rank);
  A.ctl = atc<Ctl>(h, ch, h->lay.ctl);
  A.pub = atc<uint64_t>(h, ch, h->lay.pub);
  A.chain = ch;
  A.probit = c.probit;
  A.probit_offset = c.probit_offset;
  A.latent = c.probit ? atc<float>(h, ch, h->lay.latent) : nullptr;
  A.ybin = c.probit ? at<uint8_t>(h, h->lay.ybin) : nullptr;
  A.n = c.n;
  A.p = c.p;
  A.m = c.ntree;
  A.D = c.max_depth;
  A.H = h->H;
  A.p_nz = h->p_nz;
  A.G = h->G;
  A.chunks = (int32_t)h->chunks;
  A.cpt = h->V;
  A.alpha = c.alpha;
  A.beta = c.beta;
  A.mu_mu = c.mu_mu;
  A.sigma_mu = c.sigma_mu;
  A.nu = c.nu;
  A.lambda = c.lambda;
  A.p_grow = c.p_grow;
  return A;
}

int launch_sweep(bart_handle *h, int32_t n_steps, uint64_t seed, bart_trace *trace,
                 int64_t trace_stride, bool in_scratch, uint32_t spin_limit = kSpinLimit,
                 int32_t absent_wg = -1) {
  HIP_TRY(hipSetDevice(h->device));
  // mailbox words carry launch-relative step numbers: clear both buffers of
  // every chain (a fill kernel, so the call can be captured into a graph)
  const int64_t words = 2 * (int64_t)h->G * kStride;
  if (in_scratch)
    k_clear_mailboxes<<<dim3(grid_for(words, 256), h->nchain), 256, 0, h->stream>>>(
        (char *)h->scratch_dev, 0, sizeof(uint64_t) * 2 * h->lay.gcap * kStride, words);
  else
    k_clear_mailboxes<<<dim3(grid_for(words, 256), h->nchain), 256, 0, h->stream>>>(
        h->ws, h->lay.pub, h->lay.chain_bytes, words);
  HIP_TRY(hipGetLastError());
  const SweepArgs *A = at<SweepArgs>(h, in_scratch ? h->lay.args_static : h->lay.args);
  Launch Lc{h->sweep, h->next, n_steps, seed, trace, trace_stride, spin_limit, absent_wg};
  void *args[] = {&A, &Lc};
  // the grid holds at most one workgroup per compute unit (checked at init)
  const dim3 grid(h->G * h->nchain);
  if (h->cfg.launch == BART_LAUNCH_COOPERATIVE)
    HIP_TRY(hipLaunchCooperativeKernel((const void *)h->fn, grid, dim3(kBlock), args, 0,
                                       h->stream));
  else
    HIP_TRY(hipLaunchKernel((const void *)h->fn, grid, dim3(kBlock), args, 0, h->stream));
  return BART_OK;
}

void advance(bart_handle *h, int64_t steps) {
  const int64_t per = (int64_t)h->cfg.ntree + 1;
  const int64_t pos = h->sweep * per + h->next + steps;
  h->sweep = pos / per;
  h->next = (int32_t)(pos % per);
}

// Steps in launches of at most kMaxLaunchSteps (the mailbox step numbers
// are 20 bits wide and restart with every launch).
int run_steps(bart_handle *h, int64_t steps, uint64_t seed, bart_trace *trace,
              bool in_scratch = false) {
  int64_t done = 0;
  while (done < steps) {
    const int32_t k = (int32_t)std::min<int64_t>(steps - done, kMaxLaunchSteps);
    const int rc = launch_sweep(h, k, seed, trace ? trace + done : nullptr, steps, in_scratch);
    if (rc) return rc;
    advance(h, k);
    done += k;
  }
  return BART_OK;
}

}  // namespace

extern "C" {

const char *bart_last_error(void) { return g_err.c_str(); }

size_t bart_workspace_bytes(const bart_config *cfg) {
  if (check_config(cfg)) return 0;
  return make_layout(*cfg).total;
}

int bart_init(const bart_config *cfg, const uint8_t *X_b, const float *y_c, const int32_t *n_cuts,
              void *workspace, size_t ws_bytes, void *stream, bart_handle **out) {
  if (!out) return fail(BART_EINVAL, "out is NULL");
  *out = nullptr;
  if (const char *why = check_config(cfg)) return fail(BART_EINVAL, "%s", why);
  if (!X_b || !y_c || !n_cuts || !workspace) return fail(BART_EINVAL, "NULL pointer argument");
  if ((uintptr_t)workspace % kAlign) return fail(BART_ENOSPACE, "workspace not 256-byte aligned");
  if ((uintptr_t)X_b % 16) return fail(BART_EINVAL, "X_b not 16-byte aligned");
  const Layout lay = make_layout(*cfg);
  if (ws_bytes < lay.total)
    return fail(BART_ENOSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, lay.total);
  std::vector<int32_t> nc(n_cuts, n_cuts + cfg->p), nzl, nzr(cfg->p, -1);
  for (int a = 0; a < cfg->p; ++a) {
    if (nc[a] < 0 || nc[a] > 255) return fail(BART_EINVAL, "n_cuts[%d]=%d not in [0,255]", a, nc[a]);
    if (nc[a] > 0) {
      nzr[a] = (int32_t)nzl.size();
      nzl.push_back(a);
    }
  }
  const int64_t chunks = ((int64_t)cfg->n + 3) / 4;
  int device = 0;
  HIP_TRY(hipGetDevice(&device));
  uint64_t *scratch_dev = nullptr;
  if (const int rc = scratch_ptr(device, &scratch_dev)) return rc;
  hipDeviceProp_t prop;
  HIP_TRY(hipGetDeviceProperties(&prop, device));
  // launch shape: one workgroup per CU at most, every workgroup owns a slice
  // of the observations of its chain.  Residuals in registers: the fewest
  // chunks of 4 observations per thread (V) that fit; streamed from HBM
  // otherwise.
  const int nchain = lay.nchain;
  const int gmax = std::min(prop.multiProcessorCount, kMaxGrid) / nchain;
  if (gmax < 1)
    return fail(BART_ENOTSUP, "nchain=%d exceeds the %d compute units", nchain,
                prop.multiProcessorCount);
  if (cfg->grid > gmax)
    return fail(BART_ENOTSUP, "grid=%d x nchain=%d exceeds the %d compute units", cfg->grid,
                nchain, prop.multiProcessorCount);
  int V = 0, G = 0;
  if (cfg->residency != BART_RESID_STREAMED && cfg->idx_bytes != 0) {
    for (int v : kVs) {
      const int64_t need = (chunks + (int64_t)v * kBlock - 1) / ((int64_t)v * kBlock);
      const int g = cfg->grid > 0 ? cfg->grid : (int)std::max<int64_t>(need, 1);
      if (need <= g && g <= gmax) {
        V = v;
        G = g;
        break;
      }
    }
    if (!V && cfg->residency == BART_RESID_REGISTERS)
      return fail(BART_ENOTSUP,
                  "n=%d needs more than %d workgroups x %d chunks of 4 observations in registers",
                  cfg->n, gmax, kVs[3]);
  }
  const bool streamed = !V;
  int cpt = V;
  if (streamed) {
    G = cfg->grid > 0 ? cfg->grid : gmax;
    cpt = (int)((chunks + (int64_t)G * kBlock - 1) / ((int64_t)G * kBlock));
  }
  SweepFn fn = streamed ? stream_fn(cfg->idx_bytes, cpt) : sweep_fn(V, cfg->idx_bytes);
  int per_cu = 0;
  HIP_TRY(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void *)fn, kBlock, 0));
  if (per_cu < 1) return fail(BART_ENOTSUP, "sweep kernel does not fit on a compute unit");
  hipFuncAttributes fa;
  HIP_TRY(hipFuncGetAttributes(&fa, (const void *)fn));

  bart_handle *h = new bart_handle();
  h->cfg = *cfg;
  h->lay = lay;
  h->ws = (char *)workspace;
  h->X = X_b;
  h->stream = (hipStream_t)stream;
  h->device = device;
  h->H = 1 << (cfg->max_depth - 1);
  h->p_nz = (int)nzl.size();
  h->V = cpt;
  h->streamed = streamed;
  h->G = G;
  h->nchain = nchain;
  h->lds = (int)fa.sharedSizeBytes;
  h->chunks = chunks;
  h->sweep = 0;
  h->next = 0;
  h->n_cuts = nc;
  h->nz_list = nzl;
  h->nz_rank = nzr;
  h->fn = fn;
  h->scratch_dev = scratch_dev;
  if (h->nz_list.empty()) h->nz_list.push_back(0);

  auto init = [&]() -> int {
    hipStream_t st = h->stream;
    HIP_TRY(hipMemcpyAsync(at<int32_t>(h, lay.n_cuts), h->n_cuts.data(), sizeof(int32_t) * cfg->p,
                           hipMemcpyHostToDevice, st));
    HIP_TRY(hipMemcpyAsync(at<int32_t>(h, lay.nz_list), h->nz_list.data(),
                           sizeof(int32_t) * std::min<size_t>(h->nz_list.size(), cfg->p),
                           hipMemcpyHostToDevice, st));
    HIP_TRY(hipMemcpyAsync(at<int32_t>(h, lay.nz_rank), h->nz_rank.data(), sizeof(int32_t) * cfg->p,
                           hipMemcpyHostToDevice, st));
    const int64_t entries = cfg->idx_bytes ? (int64_t)cfg->ntree * lay.n_pad : 2 * lay.n_pad;
    std::vector<SweepArgs> args(nchain);
    for (int c = 0; c < nchain; ++c) {
      k_init_resid<<<grid_for(lay.n_pad, 256), 256, 0, st>>>(atc<float>(h, c, lay.resid), y_c,
                                                               cfg->n, lay.n_pad);
      k_fill_idx<<<grid_for(entries, 256), 256, 0, st>>>(atc<uint8_t>(h, c, lay.idx), entries,
                                                           cfg->idx_bytes ? cfg->idx_bytes : 1,
                                                           cfg->n, lay.n_pad);
      k_init_trees<<<grid_for((int64_t)cfg->ntree * 2 * h->H, 256), 256, 0, st>>>(
          atc<uint16_t>(h, c, lay.axis), atc<uint8_t>(h, c, lay.cut), atc<float>(h, c, lay.leaf),
          atc<int32_t>(h, c, lay.count), cfg->ntree, h->H, cfg->n);
      if (cfg->probit)
        k_init_probit<<<grid_for(lay.n_pad, 256), 256, 0, st>>>(
            y_c, c == 0 ? at<uint8_t>(h, lay.ybin) : nullptr, atc<float>(h, c, lay.latent),
            atc<float>(h, c, lay.resid), cfg->probit_offset, cfg->n, lay.n_pad);
      k_set_ctl<<<1, 64, 0, st>>>(atc<Ctl>(h, c, lay.ctl), cfg->probit ? 1.0 : cfg->sigma2_init,
                                  0, 1);
      HIP_TRY(hipGetLastError());
      args[c] = make_args(h, c);
    }
    HIP_TRY(hipMemcpyAsync(at<SweepArgs>(h, lay.args), args.data(), sizeof(SweepArgs) * nchain,
                           hipMemcpyHostToDevice, st));
    // bart_step_static: chain c's mailboxes in its slice of the scratch array
    std::vector<SweepArgs> args_s(args);
    for (int c = 0; c < nchain; ++c)
      args_s[c].pub = h->scratch_dev + (int64_t)c * 2 * lay.gcap * kStride;
    HIP_TRY(hipMemcpyAsync(at<SweepArgs>(h, lay.args_static), args_s.data(),
                           sizeof(SweepArgs) * nchain, hipMemcpyHostToDevice, st));
    // the host copies of n_cuts must stay valid until the copies ran
    HIP_TRY(hipStreamSynchronize(st));
    return BART_OK;
  };
  const int rc = init();
  if (rc) {
    delete h;
    return rc;
  }
  *out = h;
  return BART_OK;
}

int bart_step(bart_handle *h, int32_t k_sweeps, uint64_t seed) {
  if (!h) return fail(BART_EINVAL, "handle is NULL");
  if (k_sweeps < 0) return fail(BART_EINVAL, "k_sweeps must be >= 0");
  if (h->next != 0) return fail(BART_ESTATE, "chain is inside sweep %lld (step %d)",
                                (long long)h->sweep, h->next);
  const int64_t steps = (int64_t)k_sweeps * (h->cfg.ntree + 1);
  return run_steps(h, steps, seed, nullptr);
}

int bart_step_static(bart_handle *h, int32_t k_sweeps, uint64_t seed) {
  if (!h) return fail(BART_EINVAL, "handle is NULL");
  if (k_sweeps < 0) return fail(BART_EINVAL, "k_sweeps must be >= 0");
  if (h->next != 0) return fail(BART_ESTATE, "chain is inside sweep %lld (step %d)",
                                (long long)h->sweep, h->next);
  const int64_t need = (int64_t)h->nchain * 2 * h->lay.gcap * kStride;
  if (need > kScratchWords)
    return fail(BART_ENOTSUP, "the mailboxes need %lld words, the static scratch holds %lld",
                (long long)need, (long long)kScratchWords);
  if (!h->scratch_dev) return fail(BART_ESTATE, "no static scratch address for device %d", h->device);
  const int64_t steps = (int64_t)k_sweeps * (h->cfg.ntree + 1);
  return run_steps(h, steps, seed, nullptr, true);
}

int bart_debug_steps(bart_handle *h, int32_t n_steps, uint64_t seed, bart_trace *trace) {
  if (!h) return fail(BART_EINVAL, "handle is NULL");
  if (n_steps < 0) return fail(BART_EINVAL, "n_steps must be >= 0");
  if (n_steps > 0 && !trace) return fail(BART_EINVAL, "trace is NULL");
  return run_steps(h, n_steps, seed, trace);
}

int bart_debug_stall(bart_handle *h, int32_t n_steps, uint64_t seed, int32_t wg,
                     uint32_t spin_limit) {
  if (!h) return fail(BART_EINVAL, "handle is NULL");
  if (n_steps < 1 || n_steps > kMaxLaunchSteps)
    return fail(BART_EINVAL, "n_steps must be in [1, %d]", kMaxLaunchSteps);
  if (wg < 0 || wg >= h->G * h->nchain)
    return fail(BART_EINVAL, "wg %d is not in the launch grid of %d", wg, h->G * h->nchain);
  if (spin_limit < 1) return fail(BART_EINVAL, "spin_limit must be >= 1");
  return launch_sweep(h, n_steps, seed, nullptr, 0, false, spin_limit, wg);
}

int bart_predict(bart_handle *h, const uint8_t *Xt, int64_t xt_stride, int64_t n_t, double offset,
                 float *out) {
  if (!h) return fail(BART_EINVAL, "handle is NULL");
  if (n_t < 0) return fail(BART_EINVAL, "n_t must be >= 0");
  if (n_t == 0) return BART_OK;
  if (!Xt || !out) return fail(BART_EINVAL, "NULL pointer argument");
  if (xt_stride < n_t || xt_stride % 16) return fail(BART_EINVAL, "xt_stride must be >= n_t and a multiple of 16");
  HIP_TRY(hipSetDevice(h->device));
  k_predict<false><<<dim3(grid_for(n_t, kPredBlock), h->nchain), kPredBlock, 0, h->stream>>>(
      Xt, xt_stride, n_t, h->cfg.p, atc<uint16_t>(h, 0, h->lay.axis),
      atc<uint8_t>(h, 0, h->lay.cut), atc<float>(h, 0, h->lay.leaf), h->cfg.ntree,
      h->cfg.max_depth, h->H, offset, h->lay.chain_bytes, out, nullptr, nullptr);
  HIP_TRY(hipGetLastError());
  return BART_OK;
}

int bart_predict_accumulate(bart_handle *h, const uint8_t *Xt, int64_t xt_stride, int64_t n_t,
                            double offset, double *sum, double *sumsq) {
  if (!h) return fail(BART_EINVAL, "handle is NULL");
  if (n_t < 0) return fail(BART_EINVAL, "n_t must be >= 0");
  if (n_t == 0) return BART_OK;
  if (!Xt || !sum || !sumsq) return fail(BART_EINVAL, "NULL pointer argument");
  if (xt_stride < n_t || xt_stride % 16) return fail(BART_EINVAL, "xt_stride must be >= n_t and a multiple of 16");
  if (n_t > ((int64_t)1 << 40)) return fail(BART_ENOTSUP, "n_t too large");
  HIP_TRY(hipSetDevice(h->device));
  k_predict<true><<<dim3(grid_for(n_t, kPredBlock), h->nchain), kPredBlock, 0, h->stream>>>(
      Xt, xt_stride, n_t, h->cfg.p, atc<uint16_t>(h, 0, h->lay.axis),
      atc<uint8_t>(h, 0, h->lay.cut), atc<float>(h, 0, h->lay.leaf), h->cfg.ntree,
      h->cfg.max_depth, h->H, offset, h->lay.chain_bytes, nullptr, sum, sumsq);
  HIP_TRY(hipGetLastError());
  return BART_OK;
}

int bart_posterior_summary(bart_handle *h, const double *sum, const double *sumsq, int64_t n_t,
                           int64_t n_keep, double *mean, double *sd) {
  if (!h) return fail(BART_EINVAL, "handle is NULL");
  if (n_t < 0) return fail(BART_EINVAL, "n_t must be >= 0");
  if (n_keep < 1) return fail(BART_EINVAL, "n_keep must be >= 1");
  if (n_t == 0) return BART_OK;
  if (!sum || !sumsq || !mean || !sd) return fail(BART_EINVAL, "NULL pointer argument");
  HIP_TRY(hipSetDevice(h->device));
  k_posterior_summary<<<grid_for(n_t, 256), 256, 0, h->stream>>>(sum, sumsq, n_t, h->nchain,
                                                                 1.0 / (double)n_keep, mean, sd);
  HIP_TRY(hipGetLastError());
  return BART_OK;
}

int bart_get_state(bart_handle *h, bart_state *d) {
  if (!h || !d) return fail(BART_EINVAL, "NULL argument");
  const int ch = d->chain;
  if (ch < 0 || ch >= h->nchain)
    return fail(BART_EINVAL, "chain %d not in [0, %d)", ch, h->nchain);
  HIP_TRY(hipSetDevice(h->device));
  const bart_config &c = h->cfg;
  const size_t m = c.ntree, H = h->H;
  hipStream_t st = h->stream;
  const Layout &L = h->lay;
  if (d->axis)
    HIP_TRY(hipMemcpyAsync(d->axis, atc<void>(h, ch, L.axis), 2 * m * H, hipMemcpyDeviceToDevice,
                           st));
  if (d->cut)
    HIP_TRY(hipMemcpyAsync(d->cut, atc<void>(h, ch, L.cut), m * H, hipMemcpyDeviceToDevice, st));
  if (d->leaf)
    HIP_TRY(hipMemcpyAsync(d->leaf, atc<void>(h, ch, L.leaf), 4 * m * 2 * H,
                           hipMemcpyDeviceToDevice, st));
  if (d->idx && c.idx_bytes)
    HIP_TRY(hipMemcpy2DAsync(d->idx, (size_t)c.n * c.idx_bytes, atc<void>(h, ch, L.idx),
                             (size_t)L.n_pad * c.idx_bytes, (size_t)c.n * c.idx_bytes, m,
                             hipMemcpyDeviceToDevice, st));
  if (d->idx && !c.idx_bytes) {
    // no cache: the leaves by Algorithm 1 on the current trees
    dim3 g(grid_for(c.n, 256), (unsigned)m);
    k_leaf_index<<<g, 256, 0, st>>>(h->X, c.x_stride, c.n, c.p, atc<uint16_t>(h, ch, L.axis),
                                    atc<uint8_t>(h, ch, L.cut), c.max_depth, h->H,
                                    (uint8_t *)d->idx, nullptr);
    HIP_TRY(hipGetLastError());
  }
  if (d->resid)
    HIP_TRY(hipMemcpyAsync(d->resid, atc<void>(h, ch, L.resid), 4 * (size_t)c.n,
                           hipMemcpyDeviceToDevice, st));
  if (d->count)
    HIP_TRY(hipMemcpyAsync(d->count, atc<void>(h, ch, L.count), 4 * m * 2 * H,
                           hipMemcpyDeviceToDevice, st));
  if (d->latent && c.probit)
    HIP_TRY(hipMemcpyAsync(d->latent, atc<void>(h, ch, L.latent), 4 * (size_t)c.n,
                           hipMemcpyDeviceToDevice, st));
  Ctl ctl;
  HIP_TRY(hipMemcpyAsync(&ctl, atc<void>(h, ch, L.ctl), sizeof(Ctl), hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  d->sigma2 = ctl.sigma2;
  d->sweep = h->sweep;
  d->next = h->next;
  return BART_OK;
}

int bart_set_state(bart_handle *h, const bart_state *s) {
  if (!h || !s) return fail(BART_EINVAL, "NULL argument");
  if (!s->axis || !s->cut || !s->leaf || !s->idx || !s->resid)
    return fail(BART_EINVAL, "NULL state buffer");
  const bart_config &c = h->cfg;
  const int ch = s->chain;
  if (ch < 0 || ch >= h->nchain)
    return fail(BART_EINVAL, "chain %d not in [0, %d)", ch, h->nchain);
  if (!(s->sigma2 > 0.0 && std::isfinite(s->sigma2))) return fail(BART_EINVAL, "sigma2 must be > 0");
  if (s->sweep < 0 || s->next < 0 || s->next > c.ntree) return fail(BART_EINVAL, "bad position");
  if (c.probit && !s->latent) return fail(BART_EINVAL, "a probit state needs its latents");
  HIP_TRY(hipSetDevice(h->device));
  const size_t m = c.ntree, H = h->H;
  hipStream_t st = h->stream;
  const Layout &L = h->lay;
  HIP_TRY(hipMemcpyAsync(atc<void>(h, ch, L.axis), s->axis, 2 * m * H, hipMemcpyDeviceToDevice, st));
  HIP_TRY(hipMemcpyAsync(atc<void>(h, ch, L.cut), s->cut, m * H, hipMemcpyDeviceToDevice, st));
  HIP_TRY(hipMemcpyAsync(atc<void>(h, ch, L.leaf), s->leaf, 4 * m * 2 * H, hipMemcpyDeviceToDevice,
                         st));
  if (c.idx_bytes) {
    HIP_TRY(hipMemcpy2DAsync(atc<void>(h, ch, L.idx), (size_t)L.n_pad * c.idx_bytes, s->idx,
                             (size_t)c.n * c.idx_bytes, (size_t)c.n * c.idx_bytes, m,
                             hipMemcpyDeviceToDevice, st));
    if (L.n_pad > c.n)
      k_zero_idx_pad<<<grid_for((int64_t)m * (L.n_pad - c.n), 256), 256, 0, st>>>(
          atc<uint8_t>(h, ch, L.idx), c.idx_bytes, c.n, L.n_pad, (int64_t)m);
  }
  HIP_TRY(hipMemcpyAsync(atc<void>(h, ch, L.resid), s->resid, 4 * (size_t)c.n,
                         hipMemcpyDeviceToDevice, st));
  if (c.probit)
    HIP_TRY(hipMemcpyAsync(atc<void>(h, ch, L.latent), s->latent, 4 * (size_t)c.n,
                           hipMemcpyDeviceToDevice, st));
  const int64_t cells = (int64_t)m * 2 * H;
  k_zero_i32<<<grid_for(cells, 256), 256, 0, st>>>(atc<int32_t>(h, ch, L.count), cells);
  if (c.idx_bytes) {
    dim3 g(std::min<int64_t>(((int64_t)c.n + 1023) / 1024, 64), (unsigned)m);
    k_recount<<<g, 1024, 0, st>>>(atc<uint8_t>(h, ch, L.idx), L.n_pad, c.idx_bytes,
                                  atc<int32_t>(h, ch, L.count), c.n, h->H,
                                  &atc<Ctl>(h, ch, L.ctl)->error);
  } else {
    dim3 g(grid_for(c.n, 256), (unsigned)m);
    k_leaf_index<<<g, 256, 0, st>>>(h->X, c.x_stride, c.n, c.p, atc<uint16_t>(h, ch, L.axis),
                                    atc<uint8_t>(h, ch, L.cut), c.max_depth, h->H, nullptr,
                                    atc<int32_t>(h, ch, L.count));
  }
  // the position is shared by all chains
  for (int k = 0; k < h->nchain; ++k)
    k_set_ctl<<<1, 64, 0, st>>>(atc<Ctl>(h, k, L.ctl), k == ch ? s->sigma2 : -1.0, s->sweep, 0);
  HIP_TRY(hipGetLastError());
  h->sweep = s->sweep;
  h->next = s->next;
  return BART_OK;
}

int bart_status(bart_handle *h, uint32_t *bits) {
  if (!h) return fail(BART_EINVAL, "handle is NULL");
  HIP_TRY(hipSetDevice(h->device));
  std::vector<Ctl> ctl(h->nchain);
  for (int c = 0; c < h->nchain; ++c)
    HIP_TRY(hipMemcpyAsync(&ctl[c], atc<void>(h, c, h->lay.ctl), sizeof(Ctl),
                           hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(hipStreamSynchronize(h->stream));
  uint32_t err = 0;
  for (const Ctl &x : ctl) err |= x.error;
  if (bits) *bits = err;
  if (err) return fail(BART_EDEVICE, "device error bits 0x%x", err);
  return BART_OK;
}

int bart_move_stats(bart_handle *h, int32_t chain, uint64_t *out) {
  if (!h || !out) return fail(BART_EINVAL, "NULL argument");
  if (chain < 0 || chain >= h->nchain)
    return fail(BART_EINVAL, "chain %d not in [0, %d)", chain, h->nchain);
  HIP_TRY(hipSetDevice(h->device));
  Ctl ctl;
  HIP_TRY(hipMemcpyAsync(&ctl, atc<void>(h, chain, h->lay.ctl), sizeof(Ctl), hipMemcpyDeviceToHost,
                         h->stream));
  HIP_TRY(hipStreamSynchronize(h->stream));
  for (int k = 0; k < 6; ++k) out[k] = ctl.stats[k];
  return BART_OK;
}

int bart_launch_info(const bart_handle *h, bart_launch *o) {
  if (!h || !o) return fail(BART_EINVAL, "NULL argument");
  memset(o, 0, sizeof *o);
  o->grid = h->G;
  o->block = kBlock;
  o->chunks_per_thread = h->V;
  o->residency = h->streamed ? BART_RESID_STREAMED : BART_RESID_REGISTERS;
  o->lds_bytes = h->lds;
  o->obs_per_thread = 4 * h->V;
  o->max_leaves = std::min(h->H, kMaxLeaves);
  o->launch = h->cfg.launch;
  o->nchain = h->nchain;
  o->rank_stash = h->streamed && h->V <= kStashCpt ? 1 : 0;
  o->stash_chunks = kStashCpt;
  o->lds_resid_chunks = o->rank_stash ? resid_lds_chunks(h->V) : 0;
  return BART_OK;
}

void bart_destroy(bart_handle *h) { delete h; }

#ifdef BART_PHASE_CLOCKS
// Diagnostic build only: the phase clocks of the last launch of the register
// kernel, u64 [kMaxGrid][kClockSteps][kClockPh] (see sweep.hpp), into host
// memory of `words` u64; synchronises the device.
int bart_phase_clocks(uint64_t *host, size_t words) {
  if (!host || words < (size_t)kMaxGrid * kClockSteps * kClockPh)
    return fail(BART_EINVAL, "need %zu words", (size_t)kMaxGrid * kClockSteps * kClockPh);
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpyFromSymbol(host, HIP_SYMBOL(g_phase_clock),
                              sizeof(uint64_t) * kMaxGrid * kClockSteps * kClockPh));
  return BART_OK;
}
// The stamps of the last sigma^2 step, u64 [kMaxGrid][kSigmaPh].
int bart_sigma_clocks(uint64_t *host, size_t words) {
  if (!host || words < (size_t)kMaxGrid * kSigmaPh)
    return fail(BART_EINVAL, "need %zu words", (size_t)kMaxGrid * kSigmaPh);
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpyFromSymbol(host, HIP_SYMBOL(g_sigma_clock), sizeof(uint64_t) * kMaxGrid * kSigmaPh));
  return BART_OK;
}
#endif

}  // extern "C"

// host-side input preparation (bart_cutpoints, bart_bin, bart_default_hyper)
#include "prep.hpp"
