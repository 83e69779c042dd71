// sweep.hpp -- persistent HIP kernel running whole BART sweeps on gfx950.
//
// One cooperative launch runs a range of steps; a step is the update of one
// tree (sec. 3.3, "Computations sequential along trees", items 7-11) or the
// error-variance draw that ends a sweep (sec. 3.3, "Sampling the error
// variance").  Each workgroup owns a fixed slice of the observations and
// keeps its residuals in registers for the whole launch (the residual cache
// of sec. 3.3 never leaves the chip); the index cache row of the tree being
// updated and the predictor row of its proposed axis are streamed from HBM
// (predictor-major u8, coalesced 4-byte chunks).
//
// Per tree step:
//   1. route (sec. 3.3 item 2): idx' = 2 eta + [x_a >= s] for points in the
//      grown leaf, the index otherwise; converted to the rank of the leaf in
//      the larger tree;
//   2. indexed reduce (item 7, "the bottleneck"): per-lane private LDS bins
//      of fp32 residual sums, then a fixed-order workgroup reduction in fp64;
//   3. every worker workgroup posts its per-leaf partials in its own mailbox
//      as (sequence << 32 | fp32 payload) words; no atomics, no fences;
//   4. workgroup 0 (the "master", which owns no observations) gathers the
//      mailboxes in fixed order (so the sums are deterministic), finishes the
//      MH ratio (items 8-9), draws the leaves (item 10) and posts the flags
//      and per-leaf residual deltas in one contiguous result block;
//   5. each worker polls that block with one coalesced wave load, applies
//      r += old - new (item 11) and rewrites the index row where the tree
//      changed.
// While waiting in step j every workgroup already loads the index row and
// predictor row of tree j+1: proposals do not depend on earlier trees
// (sec. 3.3, "Computations parallel across trees").
#pragma once
#include "common.hpp"
#include "propose.hpp"
#include "rng.hpp"

namespace bart {

constexpr uint32_t kSpinLimit = 1u << 21;

__device__ __forceinline__ uint64_t ld_dev(uint64_t *p) {
  return __hip_atomic_load(gbl(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(uint64_t *p, uint64_t v) {
  __hip_atomic_store(gbl(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t word(uint32_t seq, uint32_t payload) {
  return ((uint64_t)seq << 32) | payload;
}

// Bounded wait until *p carries sequence seq; false on timeout.
__device__ __forceinline__ bool wait_word(uint64_t *p, uint32_t seq, uint64_t &v) {
  v = ld_dev(p);
  uint32_t spins = 0;
  while ((uint32_t)(v >> 32) != seq) {
    __builtin_amdgcn_s_sleep(1);
    if (++spins > kSpinLimit) return false;
    v = ld_dev(p);
  }
  return true;
}

// Workgroup barrier that orders LDS accesses only: outstanding global loads
// (prefetches of the next tree) stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// One DPP move of an fp64 value (both 32-bit halves from the same lane);
// lanes whose source is disabled or out of range read 0.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, kCtrl, kRowMask, 0xF, true);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), kCtrl, kRowMask, 0xF, true);
  return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}

// Sum over the 64 lanes of a wave with DPP row shifts and row broadcasts, in
// a fixed order; the total is valid in lane 63.
__device__ __forceinline__ double wave_total63(double v) {
  v += dpp_f64<0x111, 0xF>(v);  // row_shr:1
  v += dpp_f64<0x112, 0xF>(v);  // row_shr:2
  v += dpp_f64<0x114, 0xF>(v);  // row_shr:4
  v += dpp_f64<0x118, 0xF>(v);  // row_shr:8  -> lane 15 of each row holds the row sum
  v += dpp_f64<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
  v += dpp_f64<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
  return v;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Log marginal-likelihood ratio of splitting a leaf into (L, R): the
// partial residuals of a leaf with n points, its N(mu_mu, sigma_mu^2) value
// integrated out (sec. 2.1), are N(mu_mu 1, sigma^2 I + sigma_mu^2 1 1^T).
__device__ inline double split_llr(double s2, double mu_mu, double v, double nL, double SL,
                                   double nR, double SR) {
  const double nP = nL + nR, SP = SL + SR;
  const double tL = SL - nL * mu_mu, tR = SR - nR * mu_mu, tP = SP - nP * mu_mu;
  const double qL = tL * tL / (s2 + nL * v);
  const double qR = tR * tR / (s2 + nR * v);
  const double qP = tP * tP / (s2 + nP * v);
  const double det = 0.5 * log(s2 * (s2 + nP * v) / ((s2 + nL * v) * (s2 + nR * v)));
  return det + v / (2.0 * s2) * (qL + qR - qP);
}

// Per-workgroup view of the tree being stepped.
struct Ctx {
  Prop pr;
  uint8_t rank_of[256];          // heap slot -> rank among larger-tree leaves (0xFF: none)
  uint16_t heap_of[kMaxLeaves];  // rank -> heap slot
};

struct Shared {
  float bins[kBinFloats];
  Ctx ctx[2];
  double red[kMaxLeaves + 1];
  double part[kBlock];
  double tot[2 * kMaxLeaves + 1];
  double S[kMaxLeaves];
  double cntd[kMaxLeaves];
  float mu_old[kMaxLeaves];
  float delta[kMaxLeaves];
  uint16_t fin[kMaxLeaves];
  double wave_part[kWaves];
  uint32_t res[kMaxLeaves + 1];  // master: payloads of the result boxes
  float newv[kMaxLeaves];
  bart_trace rec;
  double sigma2;
  double dec_logr, dec_S_eta, dec_n_eta;
  int red_nr;
  int flags;  // bit0 accept, bit1 merged
  int abort_flag;
  int dev_err;
};

template <int IB>
struct IdxChunk;
template <>
struct IdxChunk<1> {
  using T = uint32_t;
  static __device__ __forceinline__ int get(T c, int b) { return (c >> (8 * b)) & 0xff; }
  static __device__ __forceinline__ T put(T c, int b, int v) { return c | ((T)v << (8 * b)); }
};
template <>
struct IdxChunk<2> {
  using T = uint64_t;
  static __device__ __forceinline__ int get(T c, int b) { return (int)((c >> (16 * b)) & 0xff); }
  static __device__ __forceinline__ T put(T c, int b, int v) { return c | ((T)v << (16 * b)); }
};

// Proposal of tree j: thread t < 24 loads 32-bit word t of its record
// (a lane-varying load, so nothing waits for it until it is stored to LDS).
constexpr int kPropWords = (int)(sizeof(Prop) / 4);

__device__ __forceinline__ uint32_t load_prop_word(const SweepArgs *__restrict__ A, int j) {
  const int t = threadIdx.x;
  return t < kPropWords ? (gbl((const uint32_t *)(A->prop + j)))[t] : 0u;
}

// Rank table of the larger tree from the proposal record already in LDS.
__device__ __forceinline__ void build_ranks(const SweepArgs *__restrict__ A, Ctx &c) {
  const int t = threadIdx.x;
  if (t < 256) {
    const int h = t;
    uint8_t r = 0xFF;
    if (h < 2 * A->H && ((c.pr.mask[h >> 6] >> (h & 63)) & 1ull)) {
      int k = 0;
      for (int u = 0; u < (h >> 6); ++u) k += __popcll(c.pr.mask[u]);
      if (h & 63) k += __popcll(c.pr.mask[h >> 6] & ((1ull << (h & 63)) - 1ull));
      r = (uint8_t)k;
      c.heap_of[k] = (uint16_t)h;
    }
    c.rank_of[h] = r;
  }
}

// Leaf normals of sweep s for trees >= j0, grid-stride over (tree, pair of
// heap slots); each Philox block gives the normals of slots 2u and 2u+1.
__device__ __noinline__ void gen_normals(const SweepArgs *__restrict__ A, uint64_t seed, int64_t s,
                                         int j0) {
  const int H = A->H;
  double *zb = A->z + (int64_t)(s & 1) * A->m * 2 * H;
  const int64_t gsz = (int64_t)A->G * kBlock;
  for (int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x; q < (int64_t)A->m * H; q += gsz) {
    const int tr = (int)(q / H), u = (int)(q % H);
    if (tr < j0) continue;
    const Block bl = draw(seed, (uint64_t)s, (uint64_t)tr, 1, (uint64_t)u);
    zb[(int64_t)tr * 2 * H + 2 * u] = gauss(bl.w0, bl.w1);
    zb[(int64_t)tr * 2 * H + 2 * u + 1] = gauss(bl.w2, bl.w3);
  }
}

// Master: proposals of trees [j0, m) of sweep s, one thread per tree.
__device__ __noinline__ void gen_proposals(const SweepArgs *__restrict__ A, uint64_t seed, int64_t s,
                                           int j0) {
  for (int tr = j0 + (int)threadIdx.x; tr < A->m; tr += kBlock)
    propose_tree(A, seed, tr, s, A->prop[tr]);
}

// Master: copy the staged trace record of a step out and clear the stage.
__device__ __noinline__ void flush_trace(bart_trace *dst, bart_trace *stage) {
  uint32_t *d = (uint32_t *)dst;
  uint32_t *src = (uint32_t *)stage;
  for (int q = threadIdx.x; q < (int)(sizeof(bart_trace) / 4); q += kBlock) {
    d[q] = src[q];
    src[q] = 0u;
  }
}

// Master: sigma^2 | rest ~ InvGamma((nu+n)/2, (nu lambda + SSR)/2), the
// conjugate update of the prior lambda nu / sigma^2 ~ chi^2_nu (eq. bartdef).
__device__ __noinline__ double draw_sigma2(const SweepArgs *__restrict__ A, uint64_t seed, int64_t s,
                                           double ssr) {
  const double shape = 0.5 * (A->nu + (double)A->n);
  const double scale = 0.5 * (A->nu * A->lambda + ssr);
  return scale / gamma_mt(seed, (uint64_t)s, shape);
}

// Grid-wide rendezvous at sequence seq (prologue): every workgroup posts
// word 0 of its mailbox, the master waits for all of them and answers in
// result word 0.  Callers release their writes before, acquire after.
__device__ __forceinline__ void rendezvous(const SweepArgs *__restrict__ A, Shared &sh,
                                           uint32_t seq, bool master) {
  const int t = threadIdx.x;
  if (t == 0) st_dev(&A->slots[(int64_t)blockIdx.x * kSlot], word(seq, 0));
  if (master) {
#pragma unroll 1
    for (int g = 1 + t; g < A->G; g += kBlock) {
      uint64_t v;
      if (!wait_word(&A->slots[(int64_t)g * kSlot], seq, v)) sh.abort_flag = 1;
    }
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "agent");
    __syncthreads();
    for (int g = 1 + t; g < A->G; g += kBlock) st_dev(&A->boxes[(int64_t)g * kSlot], word(seq, 0));
  } else {
    if (t == 0) {
      uint64_t v;
      if (!wait_word(&A->boxes[(int64_t)blockIdx.x * kSlot], seq, v)) sh.abort_flag = 1;
    }
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
}

// Worker: wait until words 0..nw-1 (nw <= 64) of its own result box all
// carry seq, polling them with one coalesced load of the calling wave per
// round (the box is written by the master alone and read by this workgroup
// alone, so polls never queue behind other workgroups'); lane k returns word k.
__device__ __forceinline__ uint64_t poll_result(const SweepArgs *__restrict__ A, Shared &sh,
                                                uint32_t seq, int nw) {
  const int lane = threadIdx.x & 63;
  uint64_t v = 0;
  uint32_t spins = 0;
  while (true) {
    if (lane < nw) v = ld_dev(&A->boxes[(int64_t)blockIdx.x * kSlot + lane]);
    const bool ready = lane >= nw || (uint32_t)(v >> 32) == seq;
    if (__all(ready)) break;
    __builtin_amdgcn_s_sleep(1);
    if (++spins > kSpinLimit) {
      sh.abort_flag = 1;
      break;
    }
  }
  return v;
}

// ------------------------------------------------------------------ master
// Per-rank data of the tree about to be decided, loaded ahead of its step.
struct MasterPre {
  int h, cnt, eta_cnt;
  float leaf, eta_leaf;
  double z, eta_z;
};

// Master: proposal of tree j into ctx c, then its per-rank tree data (heap
// slot, stored count, current value, leaf normal) into registers.  Called
// right after the previous step was posted, so these loads overlap the
// workers' data pass.
__device__ __forceinline__ MasterPre master_prepare(const SweepArgs *__restrict__ A, Shared &sh,
                                                    Ctx &c, int j, int64_t s) {
  const int t = threadIdx.x, H = A->H;
  const uint32_t wd = load_prop_word(A, j);
  if (t < kPropWords) ((uint32_t *)&c.pr)[t] = wd;
  lds_barrier();
  build_ranks(A, c);
  lds_barrier();
  MasterPre m{0, 0, 0, 0.f, 0.f, 0.0, 0.0};
  const int L = c.pr.L, move = c.pr.move, eta = c.pr.eta;
  if (t < L) {
    const gptr<const float> lf = gbl((const float *)A->leaf) + (int64_t)j * 2 * H;
    const gptr<const int32_t> cn = gbl((const int32_t *)A->count) + (int64_t)j * 2 * H;
    const gptr<const double> zj =
        gbl((const double *)A->z) + ((int64_t)(s & 1) * A->m + j) * 2 * H;
    m.h = c.heap_of[t];
    m.cnt = cn[m.h];
    m.leaf = lf[m.h];
    m.z = zj[m.h];
    if (move != kNone) {
      m.eta_cnt = cn[eta];
      m.eta_leaf = lf[eta];
      m.eta_z = zj[eta];
    }
  }
  return m;
}

__device__ __forceinline__ void master_loop(const SweepArgs *__restrict__ A, const Launch &Lc,
                                            Shared &sh) {
  const int t = threadIdx.x;
  const int H = A->H;
  const bool tracing = Lc.trace != nullptr;
  const uint64_t seed = Lc.seed;
  const int Wn = A->G - 1;  // worker workgroups 1..G-1
  if (tracing)
    for (int q = t; q < (int)(sizeof(bart_trace) / 4); q += kBlock) ((uint32_t *)&sh.rec)[q] = 0u;
  if (t == 0) {
    sh.abort_flag = 0;
    sh.dev_err = 0;
    sh.sigma2 = A->ctl->sigma2;
  }
  int64_t s = Lc.s0;
  int j = Lc.j0;
  if (j < A->m) {
    gen_proposals(A, seed, s, j);
    gen_normals(A, seed, s, j);
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  rendezvous(A, sh, 1, true);
  int cb = 0;
  MasterPre pre{0, 0, 0, 0.f, 0.f, 0.0, 0.0};
  if (j < A->m) pre = master_prepare(A, sh, sh.ctx[cb], j, s);
  __syncthreads();

#pragma unroll 1
  for (int step = 0; step < Lc.n_steps; ++step) {
    if (sh.abort_flag) break;
    const uint32_t seq = (uint32_t)step + 2;
    if (j < A->m) {
      // ================= tree step j: gather, decide, post =================
      Ctx &c = sh.ctx[cb];
      const int move = c.pr.move, eta = c.pr.eta, cutv = c.pr.cut, L = c.pr.L;
      const int kl = c.pr.rank_l, kr = c.pr.rank_r;
      const double s2 = sh.sigma2, v2 = A->sigma_mu * A->sigma_mu;
      // gather: thread (seg, k) sums word k of the workers of its segment, in order,
      // polling a batch of up to 8 mailboxes with all loads in flight at once
      const int K1 = 2 * L + 1;
      int nseg = kBlock / K1;
      if (nseg > (Wn + 7) / 8) nseg = (Wn + 7) / 8;
      if (nseg < 1) nseg = 1;
      if (t < nseg * K1) {
        const int k = t % K1, seg = t / K1;
        const int g0 = 1 + (seg * Wn) / nseg, g1 = 1 + ((seg + 1) * Wn) / nseg;
        double acc = 0.0;
#pragma unroll 1
        for (int gb = g0; gb < g1; gb += 8) {
          uint64_t wv[8];
          uint32_t pending = (g1 - gb >= 8) ? 0xFFu : ((1u << (g1 - gb)) - 1u);
          uint32_t spins = 0;
          while (pending) {
#pragma unroll
            for (int u = 0; u < 8; ++u)
              if ((pending >> u) & 1u) wv[u] = ld_dev(&A->slots[(int64_t)(gb + u) * kSlot + k]);
#pragma unroll
            for (int u = 0; u < 8; ++u)
              if (((pending >> u) & 1u) && (uint32_t)(wv[u] >> 32) == seq) pending &= ~(1u << u);
            if (pending) {
              __builtin_amdgcn_s_sleep(1);
              if (++spins > kSpinLimit) {
                sh.abort_flag = 1;
                break;
              }
            }
          }
#pragma unroll
          for (int u = 0; u < 8; ++u)
            if (gb + u < g1)
              acc += (k < 2 * L) ? (double)__uint_as_float((uint32_t)wv[u])
                                 : (double)(uint32_t)wv[u];
        }
        sh.part[t] = acc;
      }
      lds_barrier();
      if (t < K1) {
        double acc = 0.0;
        for (int seg = 0; seg < nseg; ++seg) acc += sh.part[seg * K1 + t];
        sh.tot[t] = acc;
      }
      lds_barrier();
      // partial sums S_h = R_h + n_h * (old value) (sec. 3.3 item 8)
      const double nR = sh.tot[2 * L];
      if (t < L) {
        const int h = pre.h;
        const bool child = (move == kGrow) && ((h >> 1) == eta);
        const double nk = child ? ((h & 1) ? nR : (double)pre.eta_cnt - nR) : (double)pre.cnt;
        const float mo = child ? pre.eta_leaf : pre.leaf;
        sh.cntd[t] = nk;
        sh.mu_old[t] = mo;
        sh.S[t] = (sh.tot[2 * t] + sh.tot[2 * t + 1]) + nk * (double)mo;
      }
      lds_barrier();
      // accept / reject (item 9)
      if (t == 0) {
        int acc = 0, merged = 0;
        double logr = 0.0;
        if (move != kNone) {
          const double llr =
              split_llr(s2, A->mu_mu, v2, sh.cntd[kl], sh.S[kl], sh.cntd[kr], sh.S[kr]);
          logr = c.pr.c_prior + (move == kGrow ? llr : -llr);
          acc = c.pr.ln_u < logr ? 1 : 0;
          merged = (move == kGrow && !acc) || (move == kPrune && acc);
          sh.dec_S_eta = sh.S[kl] + sh.S[kr];
          sh.dec_n_eta = sh.cntd[kl] + sh.cntd[kr];
        }
        sh.dec_logr = logr;
        sh.flags = acc | (merged << 1);
      }
      lds_barrier();
      // leaf draws of the final tree (items 4, 5, 10); box word 0 holds the
      // flags, words 1..L the residual deltas
      const int flags = sh.flags, acc = flags & 1, merged = (flags >> 1) & 1;
      if (t == 0) sh.res[0] = (uint32_t)flags;
      if (t < L) {
        const int h = pre.h;
        const bool to_eta = merged && ((h >> 1) == eta);
        const double nf = to_eta ? sh.dec_n_eta : sh.cntd[t];
        const double Sf = to_eta ? sh.dec_S_eta : sh.S[t];
        const double prec = nf / s2 + 1.0 / v2;
        const double mean = (Sf / s2 + A->mu_mu / v2) / prec;
        const float mu_new = (float)(mean + (to_eta ? pre.eta_z : pre.z) / sqrt(prec));
        sh.res[1 + t] = __float_as_uint(sh.mu_old[t] - mu_new);
        sh.newv[t] = mu_new;
      }
      lds_barrier();
      // broadcast into every worker's box: word k of box g by thread (g, k)
      for (int q = t; q < Wn * (L + 1); q += kBlock) {
        const int g = 1 + q / (L + 1), k = q % (L + 1);
        st_dev(&A->boxes[(int64_t)g * kSlot + k], word(seq, sh.res[k]));
      }
      // the final tree: values and counts of its leaves, structure change
      if (t < L) {
        const int h = pre.h;
        const bool to_eta = merged && ((h >> 1) == eta);
        const int f = to_eta ? eta : h;
        const double nf = to_eta ? sh.dec_n_eta : sh.cntd[t];
        gbl(A->leaf)[(int64_t)j * 2 * H + f] = sh.newv[t];
        gbl(A->count)[(int64_t)j * 2 * H + f] = (int32_t)nf;
        if (tracing) {
          sh.rec.leaf_new[f] = sh.newv[t];
          sh.rec.count[h] = (int32_t)sh.cntd[t];
          sh.rec.sum[h] = sh.S[t];
        }
      }
      if (t == 0) {
        const gptr<uint8_t> ct = gbl(A->cut) + (int64_t)j * H;
        const gptr<uint16_t> ax = gbl(A->axis) + (int64_t)j * H;
        if (move == kGrow && acc) {
          ax[eta] = (uint16_t)c.pr.axis;
          ct[eta] = (uint8_t)cutv;
          if (2 * eta < H) ct[2 * eta] = 0;
          if (2 * eta + 1 < H) ct[2 * eta + 1] = 0;
        }
        if (move == kPrune && acc) ct[eta] = 0;
        const gptr<uint64_t> st = gbl(A->ctl->stats);
        st[0] += move == kGrow;
        st[1] += move == kPrune;
        st[2] += move == kGrow && acc;
        st[3] += move == kPrune && acc;
        st[4] += 1;
        st[5] += (uint64_t)(L - merged);
        if (tracing) {
          bart_trace &R = sh.rec;
          R.kind = 0;
          R.tree = j;
          R.sweep = s;
          R.move = move;
          R.eta = eta;
          R.axis = c.pr.axis;
          R.cut = cutv;
          R.n_grow_cand = c.pr.nG;
          R.n_prune_cand = c.pr.nP;
          R.accept = acc;
          R.n_leaves = L;
          R.log_r = sh.dec_logr;
          R.ln_u = c.pr.ln_u;
          R.sigma2 = s2;
        }
      }
      if (tracing) {
        __syncthreads();
        flush_trace(Lc.trace + step, &sh.rec);
      }
      ++j;
      // next tree: its proposal and tree data, while the workers apply and route
      if (j < A->m && step + 1 < Lc.n_steps) pre = master_prepare(A, sh, sh.ctx[cb ^ 1], j, s);
      cb ^= 1;
    } else {
      // ================= sigma^2 step (sec. 3.3, "Sampling the error variance")
      const bool more = step + 1 < Lc.n_steps;
      if (more) {
        gen_proposals(A, seed, s + 1, 0);
        gen_normals(A, seed, s + 1, 0);
      }
#pragma unroll 1
      for (int g = 1 + t; g < A->G; g += kBlock) {
        uint64_t v;
        if (!wait_word(&A->slots[(int64_t)g * kSlot], seq, v)) sh.abort_flag = 1;
        sh.part[g] = (double)__uint_as_float((uint32_t)v);
      }
      __syncthreads();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      if (t == 0) {
        double acc = 0.0;
        for (int g = 1; g < A->G; ++g) acc += sh.part[g];
        const double s2 = draw_sigma2(A, seed, s, acc);
        sh.sigma2 = s2;
        A->ctl->sigma2 = s2;
        A->ctl->sweep = s + 1;
        if (tracing) {
          sh.rec.kind = 1;
          sh.rec.tree = A->m;
          sh.rec.sweep = s;
          sh.rec.ssr = acc;
          sh.rec.sigma2 = s2;
        }
      }
      __syncthreads();
      if (tracing) flush_trace(Lc.trace + step, &sh.rec);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      __syncthreads();
      for (int g = 1 + t; g < A->G; g += kBlock) st_dev(&A->boxes[(int64_t)g * kSlot], word(seq, 0));
      j = 0;
      ++s;
      if (more) pre = master_prepare(A, sh, sh.ctx[cb], 0, s);
    }
    lds_barrier();
  }
  if (t == 0 && (sh.abort_flag || sh.dev_err))
    atomicOr(&A->ctl->error, (sh.abort_flag ? BART_DEVERR_TIMEOUT : 0u) |
                                 (sh.dev_err ? BART_DEVERR_CACHE : 0u));
}

// ------------------------------------------------------------------ workers
template <int V, int IB>
__device__ __forceinline__ void worker_loop(const SweepArgs *__restrict__ A, const Launch &Lc,
                                            Shared &sh) {
  using IC = IdxChunk<IB>;
  using ChunkT = typename IC::T;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, w = blockIdx.x;
  const int wk = w - 1;  // worker index
  const uint64_t seed = Lc.seed;

  float r[V][4];
  uint32_t rk[V];
  ChunkT rawc[V];
  uint32_t rawx[V];
  uint32_t okm[V];  // bit b: observation 4*chunk+b exists
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const int32_t ch = (wk * V + v) * kBlock + t;
    okm[v] = 0;
    r[v][0] = r[v][1] = r[v][2] = r[v][3] = 0.f;
    if (ch < A->chunks) {
      const int32_t rem = A->n - 4 * ch;
      okm[v] = rem >= 4 ? 15u : ((1u << rem) - 1u);
      const gptr<const float> q = gbl((const float *)A->resid) + 4 * (int64_t)ch;
      r[v][0] = q[0];
      r[v][1] = q[1];
      r[v][2] = q[2];
      r[v][3] = q[3];
    }
    rk[v] = 0;
    rawc[v] = 0;
    rawx[v] = 0;
  }
  for (int k = t; k < kBinFloats; k += kBlock) sh.bins[k] = 0.f;
  if (t == 0) {
    sh.abort_flag = 0;
    sh.dev_err = 0;
    sh.red_nr = 0;
  }
  int64_t s = Lc.s0;
  int j = Lc.j0;
  if (j < A->m) gen_normals(A, seed, s, j);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  rendezvous(A, sh, 1, false);

  int cb = 0;  // ctx buffer of the tree being stepped
  // proposal word (already loaded) -> LDS, rank table, then the row loads of that tree
  auto issue = [&](int tree, uint32_t wd, int buf) {
    Ctx &c = sh.ctx[buf];
    if (t < kPropWords) ((uint32_t *)&c.pr)[t] = wd;
    lds_barrier();
    build_ranks(A, c);
    const gptr<const ChunkT> row =
        gbl((const ChunkT *)((const char *)A->idx + (int64_t)tree * A->ldi * IB));
    const gptr<const uint32_t> xrow = gbl((const uint32_t *)(A->X + (int64_t)c.pr.axis * A->ldx));
#pragma unroll
    for (int v = 0; v < V; ++v)
      if (okm[v]) {
        const int32_t ch = (wk * V + v) * kBlock + t;
        rawc[v] = row[ch];
        rawx[v] = xrow[ch];
      }
  };
  if (j < A->m && !sh.abort_flag) issue(j, load_prop_word(A, j), cb);
  __syncthreads();

#pragma unroll 1
  for (int step = 0; step < Lc.n_steps; ++step) {
    if (sh.abort_flag) break;
    const uint32_t seq = (uint32_t)step + 2;
    if (j < A->m) {
      // ================= tree step j =================
      Ctx &c = sh.ctx[cb];
      const int move = c.pr.move, eta = c.pr.eta, cutv = c.pr.cut, L = c.pr.L;
      const int setbits = L <= 32 ? 6 : 4;  // 64 or 16 lane sets per wave
      const int setmask = (1 << setbits) - 1;
      const int grow_eta = move == kGrow ? eta : -1;
      const bool next_tree = (j + 1 < A->m) && (step + 1 < Lc.n_steps);
      // 1. route (branch-free) and 2. per-lane bins
      int nr = 0;
      uint32_t bad = 0;
#pragma unroll
      for (int v = 0; v < V; ++v) {
        uint32_t pk = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int ci = IC::get(rawc[v], b);
          const int xi = (rawx[v] >> (8 * b)) & 0xff;
          const uint32_t ok = (okm[v] >> b) & 1u;
          const int in = ci == grow_eta;
          const int right = xi >= cutv;
          const int cp = in ? 2 * eta + right : ci;
          const int r0 = c.rank_of[cp & 255];
          bad |= ok & (r0 == 0xFF);
          // padding observations and (invalid) non-leaf indices use rank 0
          const int rnk = (ok && r0 != 0xFF) ? r0 : 0;
          nr += __popcll(__ballot(ok && in && right));
          pk |= (uint32_t)rnk << (8 * b);
          // bins are private: a plain read-modify-write (LDS float atomics
          // serialise across lanes and are many times slower).  With 16 lane
          // sets, lanes l, l+16, l+32, l+48 share a set and take turns.
          float &bin = sh.bins[((rnk * kWaves + wave) << setbits) | (lane & setmask)];
          const float add = ok ? r[v][b] : 0.f;
          if (setbits == 6) {
            bin += add;
          } else {
#pragma unroll
            for (int g = 0; g < 4; ++g)
              if ((lane >> 4) == g) bin += add;
          }
        }
        rk[v] = pk;
      }
      // next tree's proposal word: loaded after the route so that the wait for
      // this step's row data does not also wait for it
      const uint32_t nxt = next_tree ? load_prop_word(A, j + 1) : 0u;
      if (bad) sh.dev_err = 1;
      if (lane == 0 && nr) atomicAdd(&sh.red_nr, nr);
      lds_barrier();
      // 3. fixed-order workgroup reduction, bins zeroed for the next step
      for (int k = wave; k < L; k += kWaves) {
        double acc = 0.0;
        if (lane <= setmask) {
#pragma unroll
          for (int u = 0; u < kWaves; ++u) {
            const int q = ((k * kWaves + u) << setbits) | lane;
            acc += (double)sh.bins[q];
            sh.bins[q] = 0.f;
          }
        }
        const double tot = wave_total63(acc);
        if (lane == 63) sh.red[k] = tot;
      }
      lds_barrier();
      // each partial as an fp32 (hi, lo) pair: hi + lo carries ~48 bits of the fp64 sum
      if (t < 2 * L) {
        const double x = sh.red[t >> 1];
        const float hi = (float)x;
        const float part = (t & 1) ? (float)(x - (double)hi) : hi;
        st_dev(&A->slots[(int64_t)w * kSlot + t], word(seq, __float_as_uint(part)));
      }
      if (t == 2 * L) {
        st_dev(&A->slots[(int64_t)w * kSlot + t], word(seq, (uint32_t)sh.red_nr));
        sh.red_nr = 0;  // next added to after several barriers
      }
      // prefetch the next tree while the master decides
      if (next_tree) issue(j + 1, nxt, cb ^ 1);
      // 5. fetch flags and deltas, update residuals and the index row
      if (wave == 0) {
        const uint64_t v = poll_result(A, sh, seq, L + 1 < 64 ? L + 1 : 64);
        if (lane == 0) sh.flags = (int)(uint32_t)v;
        if (lane >= 1 && lane <= L) sh.delta[lane - 1] = __uint_as_float((uint32_t)v);
        if (L + 1 > 64) {
          // more than 63 leaves: the remaining deltas, already posted (seq checked)
          for (int k = 64 + lane; k <= L; k += 64) {
            uint64_t u;
            if (!wait_word(&A->boxes[(int64_t)w * kSlot + k], seq, u)) sh.abort_flag = 1;
            sh.delta[k - 1] = __uint_as_float((uint32_t)u);
          }
        }
      }
      lds_barrier();
      const int acc = sh.flags & 1, merged = (sh.flags >> 1) & 1;
      if (t < L) {
        const int h = c.heap_of[t];
        sh.fin[t] = (uint16_t)((merged && (h >> 1) == eta) ? eta : h);
      }
      lds_barrier();
      const bool changed = acc && move != kNone;
      const int kl = c.pr.rank_l, kr = c.pr.rank_r;
      const gptr<ChunkT> row = gbl((ChunkT *)((char *)A->idx + (int64_t)j * A->ldi * IB));
#pragma unroll
      for (int v = 0; v < V; ++v) {
        bool touch = false;
        ChunkT out = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int rnk = (rk[v] >> (8 * b)) & 0xff;
          const float d = sh.delta[rnk];
          r[v][b] += ((okm[v] >> b) & 1u) ? d : 0.f;
          touch |= (rnk == kl) || (rnk == kr);
          out = IC::put(out, b, sh.fin[rnk]);
        }
        if (changed && touch && okm[v]) row[(wk * V + v) * kBlock + t] = out;
      }
      cb ^= 1;
      ++j;
    } else {
      // ================= sigma^2 step: partial sum of squared residuals
      double ssr = 0.0;
#pragma unroll
      for (int v = 0; v < V; ++v)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const double x = ((okm[v] >> b) & 1u) ? (double)r[v][b] : 0.0;
          ssr += x * x;
        }
      ssr = wave_total63(ssr);
      if (lane == 63) sh.wave_part[wave] = ssr;
      const bool more = step + 1 < Lc.n_steps;
      if (more) gen_normals(A, seed, s + 1, 0);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      __syncthreads();
      if (t == 0) {
        double acc = 0.0;
        for (int u = 0; u < kWaves; ++u) acc += sh.wave_part[u];
        st_dev(&A->slots[(int64_t)w * kSlot], word(seq, __float_as_uint((float)acc)));
        uint64_t v;
        if (!wait_word(&A->boxes[(int64_t)w * kSlot], seq, v)) sh.abort_flag = 1;
      }
      __syncthreads();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      j = 0;
      ++s;
      if (more) issue(0, load_prop_word(A, 0), cb);
    }
    lds_barrier();
  }

  // ---- epilogue: residuals back to HBM, device errors
#pragma unroll
  for (int v = 0; v < V; ++v)
    if (okm[v]) {
      const int32_t ch = (wk * V + v) * kBlock + t;
      const gptr<float> q = gbl(A->resid) + 4 * (int64_t)ch;
      q[0] = r[v][0];
      q[1] = r[v][1];
      q[2] = r[v][2];
      q[3] = r[v][3];
    }
  if (t == 0 && (sh.abort_flag || sh.dev_err))
    atomicOr(&A->ctl->error, (sh.abort_flag ? BART_DEVERR_TIMEOUT : 0u) |
                                 (sh.dev_err ? BART_DEVERR_CACHE : 0u));
}

template <int V, int IB>
__global__ void __launch_bounds__(kBlock) sweep_kernel(const SweepArgs *__restrict__ A, Launch Lc) {
  __shared__ Shared sh;
  if (blockIdx.x == 0)
    master_loop(A, Lc, sh);
  else
    worker_loop<V, IB>(A, Lc, sh);
}

}  // namespace bart
