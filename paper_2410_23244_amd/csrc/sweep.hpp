// sweep.hpp -- persistent HIP kernel running whole BART sweeps on gfx950.
//
// One launch runs a range of steps; a step is the update of one tree (sec.
// 3.3, "Computations sequential along trees", items 7-11) or the
// error-variance draw that ends a sweep (sec. 3.3, "Sampling the error
// variance").  Every workgroup owns a fixed slice of the observations and
// keeps its residuals in registers for the whole launch (the residual cache
// of sec. 3.3 never leaves the chip); the index cache row of the tree being
// updated and the predictor row of its proposed axis are streamed from HBM
// (predictor-major u8, coalesced 4-byte chunks).
//
// There is no coordinating workgroup.  Per tree step j, every workgroup
//   1. has its per-leaf partial residual sums of tree j (and, for a GROW,
//      the count of its points going right) in its own mailbox, as 64-bit
//      words carrying a 20-bit step number over a 44-bit payload, so a
//      reader needs no fence and no separate flag (posted by the waves that
//      formed them at the end of the previous step; the streamed kernel
//      posts them at the start of the step);
//   2. routes its points through tree j+1 (the route depends only on the
//      index cache and the proposal, sec. 3.3 "Computations parallel across
//      trees") while the other mailboxes fill;
//   3. reads all mailboxes in one fixed order and sums them in fp64, so every
//      workgroup holds bit-identical totals; from them it computes the MH
//      decision (item 9) and the leaf draws (item 10) itself: the same code
//      on the same inputs gives the same result everywhere;
//   4. applies r += old - new to its residuals and rewrites its part of the
//      index row where the tree changed (item 11);
//   5. accumulates tree j+1's partial sums from the updated residuals in
//      per-lane private LDS bins and reduces them in a fixed order; the wave
//      that forms a total posts it (item 1 of step j+1).
// One cross-workgroup hop per tree.  Tree j's structure, leaf values and
// counts are written by its owner workgroup (j mod G) and read by all in
// the next sweep; the sigma^2 step publishes them with release/acquire
// fences.
#pragma once
#include "common.hpp"
#include "propose.hpp"
#include "rng.hpp"

namespace bart {

// Poll rounds a cross-workgroup wait may take before the launch gives up
// (BART_DEVERR_TIMEOUT); launches pass it in Launch::spin_limit.
constexpr uint32_t kSpinLimit = 1u << 21;

// Phase clocks (diagnostic build, -DBART_PHASE_CLOCKS, read by
// bart_phase_clocks): thread 0 of every workgroup of the register kernel
// stamps the wall clock (100 MHz) at the phase boundaries of the tree steps
// kClockStart .. kClockStart + kClockSteps - 1 of a launch, and every
// workgroup counts the mailbox loads its polls issue in each of them; the
// last thread of the workgroup (a polling thread) stamps the end of its
// reduce, the start and end of its route, its loads, and the start and the
// end of its polls.  The ordinary build compiles none of it.
constexpr int kClockStart = 205, kClockSteps = 48, kClockPh = 20;
#ifdef BART_PHASE_CLOCKS
__device__ uint64_t g_phase_clock[kMaxGrid][kClockSteps][kClockPh];
__shared__ uint64_t clk_lds[kClockSteps][kClockPh];
__device__ __forceinline__ int clock_slot(int step) {
  return step >= kClockStart && step < kClockStart + kClockSteps ? step - kClockStart : -1;
}
#define BART_CLOCK(slot, ph)                                                              \
  do {                                                                                    \
    if (threadIdx.x == 0 && (slot) >= 0) clk_lds[slot][ph] = wall_clock64();              \
  } while (0)
#define BART_CLOCK_LAST(slot, ph)                                                         \
  do {                                                                                    \
    if (threadIdx.x == kBlock - 1 && (slot) >= 0) clk_lds[slot][ph] = wall_clock64();     \
  } while (0)
#define BART_POLL_COUNT(n) (poll_loads += (n))
// the sigma^2 step: stamps of the last one of a launch, thread 0 of every
// workgroup, straight to device memory
constexpr int kSigmaPh = 9;
__device__ uint64_t g_sigma_clock[kMaxGrid][kSigmaPh];
#define BART_SCLOCK(ph)                                                           \
  do {                                                                            \
    if (threadIdx.x == 0) g_sigma_clock[blockIdx.x][ph] = wall_clock64();         \
  } while (0)
#else
__device__ __forceinline__ constexpr int clock_slot(int) { return -1; }
#define BART_CLOCK(slot, ph) \
  do {                       \
  } while (0)
#define BART_CLOCK_LAST(slot, ph) \
  do {                            \
  } while (0)
#define BART_POLL_COUNT(n) ((void)0)
#define BART_SCLOCK(ph) \
  do {                  \
  } while (0)
#endif
constexpr int kNullRank = kMaxLeaves;  // rank of a padding point (slot 0): no bin, zero delta
constexpr int kBadRank = 255;          // rank of any other non-leaf slot: likewise, and flagged
constexpr int kRing = 4;  // proposal contexts in flight: decide j, route j+1, rows j+2, load j+3
// Ranks per pass of the streamed kernel's LDS bins, one bin per lane and chunk
// position (16).
constexpr int kSlotRanks = kBinFloats / (4 * kBlock);
// The streamed kernel with a rank stash: bins for 8 ranks per pass, one per
// lane and kStashPos chunk positions; after them one 32-bit word per chunk of
// every thread (the ranks of the chunk's 4 points), and in what remains of
// the bin array the residuals of a thread's first chunks for the launch.
constexpr int kStashRanks = kSlotRanks / 2;                       // 8
constexpr int kStashPos = 2;  // n = 1e7: 1 position 211, 2 214.5, 4 207 sweeps/s
constexpr int kStashOffset = kStashRanks * kStashPos * kBlock;    // floats of bins before it
constexpr int kStashCpt = (kBinFloats - kStashOffset) / kBlock;  // chunks per thread it holds (48)
// chunks per thread (of cpt) whose residuals stay in LDS with the stash
__host__ __device__ constexpr int resid_lds_chunks(int cpt) {
  return cpt > kStashCpt ? 0
                         : (kBinFloats - kStashOffset - cpt * kBlock) / (4 * kBlock) < cpt
                               ? (kBinFloats - kStashOffset - cpt * kBlock) / (4 * kBlock)
                               : cpt;
}
static_assert(kMaxLeaves % kSlotRanks == 0 && kMaxLeaves % kStashRanks == 0,
              "the null rank must fall outside every bin pass");

__device__ __forceinline__ uint64_t ld_dev(const uint64_t *p) {
  return __hip_atomic_load(gbl(const_cast<uint64_t *>(p)), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(uint64_t *p, uint64_t v) {
  __hip_atomic_store(gbl(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Mailbox word: step number (20 bits) over a 44-bit payload.  An fp64 value
// is carried as its top 44 bits (sign, exponent, 32 mantissa bits), a count
// as an integer.
constexpr int kPayloadBits = 44;
constexpr uint64_t kPayloadMask = (1ull << kPayloadBits) - 1ull;
__device__ __forceinline__ uint64_t mk_word(uint32_t seq, uint64_t payload) {
  return ((uint64_t)seq << kPayloadBits) | payload;
}
__device__ __forceinline__ uint32_t seq_of(uint64_t w) { return (uint32_t)(w >> kPayloadBits); }
__device__ __forceinline__ uint64_t pack_f64(double x) {
  return (uint64_t)__double_as_longlong(x) >> (64 - kPayloadBits);
}
__device__ __forceinline__ double unpack_f64(uint64_t w) {
  return __longlong_as_double((long long)((w & kPayloadMask) << (64 - kPayloadBits)));
}

// Make this workgroup's writes visible at agent scope before thread 0 posts
// the word that announces them: the barrier orders every wave's writes
// before wave 0 (they reach the XCD's L2 by the workgroup-scope release it
// contains), then one agent-scope release by wave 0 writes the L2 back.  A
// release by every wave queues eight write-backs per workgroup on the XCD's
// L2 at once, and loads issued meanwhile (the proposals of the sigma^2 step)
// wait behind them.
__device__ __forceinline__ void publish_workgroup() {
  __syncthreads();
  if (threadIdx.x < 64) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
}

// Workgroup barrier that orders LDS accesses only: outstanding global loads
// (prefetches of later trees) stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Wait for every outstanding vector memory operation of this wave, as an
// instruction the compiler's own wait analysis sees.  Vector stores count in
// the same counter as loads, so after the step's stores (index row, mailbox
// words) the compiler, unable to count them through loops, would otherwise
// wait for all of them before the next use of an earlier load; issued where
// only loads are outstanding, this lets later uses go without a wait.
__device__ __forceinline__ void wait_vm_loads() {
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0), expcnt and lgkmcnt unconstrained
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


// wave_total63 of three values at once, the steps interleaved so that the
// three DPP chains overlap.
__device__ __forceinline__ void wave_totals3(double &a, double &b, double &c) {
#define BART_STEP3(ctrl, mask)        \
  a += dpp_f64<ctrl, mask>(a);        \
  b += dpp_f64<ctrl, mask>(b);        \
  c += dpp_f64<ctrl, mask>(c);
  BART_STEP3(0x111, 0xF)
  BART_STEP3(0x112, 0xF)
  BART_STEP3(0x114, 0xF)
  BART_STEP3(0x118, 0xF)
  BART_STEP3(0x142, 0xA)
  BART_STEP3(0x143, 0xC)
#undef BART_STEP3
}

// Per-workgroup view of one tree's proposal.
struct Ctx {
  Prop pr;
  uint8_t rank_of[256];   // heap slot -> rank among larger-tree leaves (kNullRank: slot 0,
                          // kBadRank: another non-leaf)
  uint16_t heap_of[256];  // rank -> heap slot; 0 from kNullRank on
  uint16_t ax[kMaxLeaves];       // without an index cache: the tree's axis and cut per
  uint8_t ct[kMaxLeaves];        // internal heap slot, for Algorithm 1
};

// Without an index cache: the internal nodes of a tree snapshot, by ring slot.
struct NodeList {
  uint64_t imask;            // internal heap slots below 64
  uint16_t axis8[8];         // axis and cut of the first 8 internal nodes
  uint8_t cut8[8];
  uint8_t nidx[kMaxLeaves];  // heap slot -> index among the internal nodes (kNoNode: none)
  uint8_t nh[kMaxLeaves];    // heap slot of the k-th internal node, in heap order
  int32_t ni;                // internal nodes
};
constexpr int kNoNode = 255;

// What the decision of one tree needs besides the sums: per rank of the
// larger tree its stored count, current value and leaf normal, and the same
// for the node eta of the move (sec. 3.3 items 4-5, 8).
struct TreeData {
  int32_t cnt[kMaxLeaves];
  float mu[kMaxLeaves];
  double z[kMaxLeaves];
  int32_t eta_cnt;
  float eta_mu;
  double eta_z;
};

struct Shared {
  alignas(16) float bins[kBinFloats];
  Ctx ctx[kRing];
  TreeData td[2];
  double part[kBlock];
  double tot[kMaxLeaves + 1];
  double S[kMaxLeaves];
  double cntd[kMaxLeaves];
  float newv[kMaxLeaves];      // new value of each larger-tree leaf if it stays a leaf
  float dlt[256];              // its residual delta: old value - new value; 0 from kNullRank on
  float newv_m;                // new value of eta if the move ends merged
  double wave_part[kWaves];
  uint64_t solo[kMaxLeaves + 1];  // one workgroup per chain: its own mailbox words
  double sigma2;
  double sig_gamma;  // Gamma((nu+n)/2, 1) variate of the next sigma^2 draw
  double dec_logr;
  // constants of tree j's decision that do not depend on its sums, computed
  // while the mailboxes fill: per rank of a leaf whose count is known, the new
  // value is S la + lb and S = R + lnm; the merged leaf likewise (ma, mb);
  // for a PRUNE, the count-only parts of the likelihood ratio
  double la[kMaxLeaves], lb[kMaxLeaves], lnm[kMaxLeaves];
  double ma, mb, pdet, pdL, pdR, pdP, gs2eP, lgs2eP;
  uint64_t stats[6];  // workgroup 0: move statistics of this launch
  int nr[2];  // GROW right-counts of the trees being routed, by tree parity
  int flags;  // bit0 accept, bit1 merged
  int abort_flag;
  int dev_err;
  NodeList nl[kRing];  // last, so the other members keep their offsets
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

constexpr int kPropWords = (int)(sizeof(Prop) / 4);

// Word t mod 24 of tree j's proposal record: a lane-varying load, so nothing
// waits for it until it is stored to LDS.  Every thread loads (a register
// that is either loaded or set would make the compiler wait for all
// outstanding loads before setting it).
__device__ __forceinline__ uint32_t load_prop_word(const SweepArgs *__restrict__ A, int j) {
  return (gbl((const uint32_t *)(A->prop + j)))[threadIdx.x % kPropWords];
}

// Rank-table entry of heap slot h of the larger tree, from the proposal
// record already in LDS; the calling lane must be h mod 64.
__device__ __forceinline__ void build_rank_slot(const SweepArgs *__restrict__ A, Ctx &c, int h) {
  uint8_t r = h == 0 ? kNullRank : kBadRank;
  if (h < 2 * A->H && ((c.pr.mask[h >> 6] >> (h & 63)) & 1ull)) {
    int k = 0;
    for (int u = 0; u < (h >> 6); ++u) k += __popcll(c.pr.mask[u]);
    // leaves below h in its 64-slot word: h & 63 is this lane
    const uint64_t mw = c.pr.mask[h >> 6];
    k += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mw >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)mw, 0u));
    r = (uint8_t)k;
    c.heap_of[k] = (uint16_t)h;
  }
  c.rank_of[h] = r;
}

// Rank table of the larger tree: threads 0..255, one slot each.
__device__ __forceinline__ void build_ranks(const SweepArgs *__restrict__ A, Ctx &c) {
  if (threadIdx.x < 256) build_rank_slot(A, c, (int)threadIdx.x);
}

// Without an index cache: the internal nodes of the tree snapshot in c (cut
// nonzero; a slot outside the tree has cut 0), numbered in heap order by a
// ballot per 64 slots.  Wave 4 (it holds no rank slot), after the snapshot
// is in LDS.
__device__ __forceinline__ void build_inodes(const SweepArgs *__restrict__ A, const Ctx &c,
                                             NodeList &nl) {
  const int t = (int)threadIdx.x, lane = t & 63;
  if ((t >> 6) != 4) return;
  const int H = A->H;
  int base = 0;
  for (int h0 = 0; h0 < H; h0 += 64) {
    const int h = h0 + lane;
    const bool in = h >= 1 && h < H && c.ct[h] != 0;
    const uint64_t bal = __ballot(in);
    const int k = base + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                       __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
    if (h < H) nl.nidx[h] = in ? (uint8_t)k : (uint8_t)kNoNode;
    if (in) nl.nh[k] = (uint8_t)h;
    if (in && k < 8) {
      nl.axis8[k] = c.ax[h];
      nl.cut8[k] = c.ct[h];
    }
    if (h0 == 0 && lane == 0) nl.imask = bal;
    base += __popcll(bal);
  }
  if (lane == 0) nl.ni = base;
}

// Thread that loads and stages the decision data of the move's node eta: in
// wave 3, which neither polls nor holds a rank (ranks are below kMaxLeaves).
constexpr int kEtaThread = 255;
static_assert(kEtaThread >= kMaxLeaves && kEtaThread < 256, "eta thread");

// Per-thread registers of one tree's decision data in flight (thread t holds
// rank t; thread kEtaThread the node eta).
struct TdRegs {
  int32_t cnt;
  float mu;
  double z;
};

__device__ __forceinline__ TdRegs load_tree_data(const SweepArgs *__restrict__ A, const Ctx &c,
                                                 int j, int64_t s) {
  const int t = threadIdx.x, H = A->H;
  // every thread loads (slot 1 when it has no rank), see load_prop_word
  int h = 1;
  if (t < c.pr.L) h = c.heap_of[t];
  if (t == kEtaThread && c.pr.move != kNone) h = c.pr.eta;
  const int64_t o = (int64_t)j * 2 * H + h;
  TdRegs r;
  r.cnt = gbl((const int32_t *)A->count)[o];
  r.mu = gbl((const float *)A->leaf)[o];
  r.z = gbl((const double *)A->z)[(int64_t)(s & 1) * A->m * 2 * H + o];
  return r;
}

__device__ __forceinline__ void store_tree_data(TreeData &td, const Ctx &c, const TdRegs &r) {
  const int t = threadIdx.x;
  if (t < c.pr.L) {
    td.cnt[t] = r.cnt;
    td.mu[t] = r.mu;
    td.z[t] = r.z;
  }
  if (t == kEtaThread) {
    td.eta_cnt = r.cnt;
    td.eta_mu = r.mu;
    td.eta_z = r.z;
  }
}

// Leaf normals of sweep s for trees >= j0, spread over every workgroup of
// the chain: item q (tree q / H and pair u = q mod H of heap slots; one
// Philox block gives the normals of slots 2u and 2u+1) goes to thread
// first + q / G of workgroup q mod G.  The threads are those of the waves
// that propose no tree (the first ceil(m / G) of a workgroup propose, see
// gen_proposals) and draw no gamma variate (the last), so the normals run
// beside the proposals on other SIMDs; with no such wave every thread takes
// part.
__device__ __noinline__ void gen_normals(const SweepArgs *__restrict__ A, uint64_t seed, int64_t s,
                                         int j0) {
  const Key key = chain_key(seed, A->chain);
  const int H = A->H, G = A->G, t = threadIdx.x;
  int first = 64 * ((A->m + G - 1) / G), last = kBlock - 64;
  if (first >= last) first = 0, last = kBlock;
  if (t < first || t >= last) return;
  double *zb = A->z + (int64_t)(s & 1) * A->m * 2 * H;
  const int64_t items = (int64_t)A->m * H;
  const int64_t stride = (int64_t)(last - first) * G;
  for (int64_t q = (int64_t)(t - first) * G + wg_id(A); q < items; q += stride) {
    const int tr = (int)(q / H), u = (int)(q % H);
    if (tr < j0) continue;
    const Block bl = draw(key, (uint64_t)s, (uint64_t)tr, 1, (uint64_t)u);
    zb[(int64_t)tr * 2 * H + 2 * u] = gauss(bl.w0, bl.w1);
    zb[(int64_t)tr * 2 * H + 2 * u + 1] = gauss(bl.w2, bl.w3);
  }
}

// Proposals of sweep s for the trees >= j0 this workgroup owns (tree j is
// owned by workgroup j mod G), one wave per tree.
__device__ __noinline__ void gen_proposals(const SweepArgs *__restrict__ A, uint64_t seed, int64_t s,
                                           int j0) {
  const Key key = chain_key(seed, A->chain);
  const int wv = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  for (int tr = wg_id(A) + A->G * wv; tr < A->m; tr += A->G * kWaves)
    if (tr >= j0) propose_tree(A, key, tr, s, A->prop[tr]);
}

// sigma^2 | rest ~ InvGamma((nu+n)/2, (nu lambda + SSR)/2), the conjugate
// update of the prior lambda nu / sigma^2 ~ chi^2_nu (eq. bartdef), drawn as
// scale / g with g ~ Gamma((nu+n)/2, 1).  g depends only on the random
// stream of sweep s, so it is drawn before the SSR is known.
__device__ __noinline__ double sigma2_gamma(const SweepArgs *__restrict__ A, uint64_t seed,
                                            int64_t s) {
  const Key key = chain_key(seed, A->chain);
  return gamma_mt(key, (uint64_t)s, 0.5 * (A->nu + (double)A->n));
}
__device__ __forceinline__ double sigma2_of(const SweepArgs *__restrict__ A, double ssr,
                                            double g) {
  return 0.5 * (A->nu * A->lambda + ssr) / g;
}

// Probit latent of one observation (sec. 5 "Mild limitations"; Albert and
// Chib 1993): z ~ N(f, 1) truncated to z > 0 (y = 1) or z <= 0 (y = 0), by
// inversion on the allowed side, stored in f32 on that side; the residual
// moves with it, r = z - f.  Returns (new z, new r).  Not inlined: the
// normal cdf and its inverse are long, and this runs once per sweep.
__device__ __noinline__ float2 latent_update(double u, uint32_t y, float z, float r) {
  const double f = (double)z - (double)r;
  double p = u * normcdf(y ? f : -f);
  p = p < 1e-300 ? 1e-300 : p;
  float zn = (float)(y ? f - normcdfinv(p) : f + normcdfinv(p));
  if (y && !(zn > 0.f)) zn = 1.17549435e-38f;  // smallest normal f32
  if (!y && zn > 0.f) zn = 0.f;
  return make_float2(zn, (float)((double)zn - f));
}

// Latents of the 4 observations of chunk ch (those set in ok) after sweep s:
// one Philox block (s, 2^64 - 2, 3, chunk) per chunk, word b for point b.
__device__ __forceinline__ void latent_chunk(const SweepArgs *__restrict__ A, uint64_t seed,
                                             int64_t s, int32_t ch, uint32_t ok, float (&r)[4]) {
  const gptr<float> zp = gbl(A->latent) + 4 * (int64_t)ch;
  const uint32_t yb = gbl((const uint32_t *)A->ybin)[ch];
  const Block bl = draw(chain_key(seed, A->chain), (uint64_t)s, ~1ull, 3, (uint64_t)ch);
  const uint64_t wd[4] = {bl.w0, bl.w1, bl.w2, bl.w3};
  float z[4] = {zp[0], zp[1], zp[2], zp[3]};
#pragma unroll
  for (int b = 0; b < 4; ++b)
    if ((ok >> b) & 1u) {
      const float2 zr = latent_update(unit(wd[b]), (yb >> (8 * b)) & 1u, z[b], r[b]);
      z[b] = zr.x;
      r[b] = zr.y;
    }
#pragma unroll
  for (int b = 0; b < 4; ++b) zp[b] = z[b];
}

// Post words 0..K-1 (this workgroup's mailbox in buffer par).
__device__ __forceinline__ uint64_t *mailbox(const SweepArgs *__restrict__ A, int par, int g) {
  return A->pub + ((int64_t)par * A->G + g) * kStride;
}

// Word k of this workgroup's mailbox in buffer par.  A chain of one
// workgroup keeps it in LDS instead: the gather reads it back unchanged, so
// the totals are bit-identical, without a round trip through device memory.
template <class SH>
__device__ __forceinline__ void post(const SweepArgs *__restrict__ A, SH &sh, int par, int k,
                                     uint64_t word) {
  if (A->G == 1)
    sh.solo[k] = word;
  else
    st_dev(mailbox(A, par, wg_id(A)) + k, word);
}

// Poll word k < K of every mailbox of buffer par until all carry step number
// seq.  The workgroups are split into nseg segments of 8 nb consecutive
// workgroups, nb the fewest batches of 8 that let nseg * K threads cover
// them; thread (seg, k) sums word k of its segment in increasing workgroup
// order in fp64 into sh.part[seg * K + k] (words k < nsum are fp64 values,
// the others counts), with all loads of a batch in flight at once.  The
// partition depends only on G and K, so every workgroup sums in the same
// order.  The polling threads are the last ceil(nseg K / 64) waves of the
// workgroup (polling thread i is thread kBlock - 64 ceil(nseg K / 64) + i):
// the waves that build no rank table and compute no constants before the
// gather, so they start polling soonest.  Returns nseg.  Ends with an LDS
// barrier.
template <class SH>
__device__ __forceinline__ int gather_polls(const SweepArgs *__restrict__ A, SH &sh, int par,
                                            uint32_t seq, int K, int nsum, uint32_t limit,
                                            int clk = -1) {
  const int G = A->G;
#ifdef BART_PHASE_CLOCKS
  uint32_t poll_loads = 0;
#endif
  if (G == 1) {
    const int t = threadIdx.x;
    lds_barrier();  // the words were staged by the waves that formed them
    if (t < K) {
      const uint64_t wv = sh.solo[t];
      double acc = 0.0;
      acc += t < nsum ? unpack_f64(wv) : (double)(wv & kPayloadMask);
      sh.part[t] = acc;
    }
    lds_barrier();
    return 1;
  }
  int nb = 1;
  while (K * ((G + 8 * nb - 1) / (8 * nb)) > kBlock) ++nb;
  const int span = 8 * nb;
  const int nseg = (G + span - 1) / span;  // nseg * K <= kBlock
  const int first = kBlock - (nseg * K + 63) / 64 * 64;  // first polling thread
  const int t = (int)threadIdx.x - first;
  BART_CLOCK_LAST(clk, 17);
  if (t >= 0 && t < nseg * K) {
    const int k = t % K, seg = t / K;
    const int g0 = seg * span, g1 = min(G, g0 + span);
    const uint64_t *base = A->pub + (int64_t)par * A->G * kStride + k;
    double acc = 0.0;
#pragma unroll 1
    for (int gb = g0; gb < g1; gb += 8) {
      uint64_t wv[8];
      uint32_t pending = (g1 - gb >= 8) ? 0xFFu : ((1u << (g1 - gb)) - 1u);
      uint32_t spins = 0;
      const uint64_t *pb = base + (int64_t)gb * kStride;
      while (pending) {
        BART_POLL_COUNT(__popc(pending));
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if ((pending >> u) & 1u) wv[u] = ld_dev(pb + u * kStride);
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (((pending >> u) & 1u) && seq_of(wv[u]) == seq) pending &= ~(1u << u);
        if (pending) {
          __builtin_amdgcn_s_sleep(1);
          if (++spins > limit) {
            sh.abort_flag = 1;
            break;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (gb + u < g1)
          acc += k < nsum ? unpack_f64(wv[u]) : (double)(wv[u] & kPayloadMask);
    }
    sh.part[t] = acc;
  }
  BART_CLOCK_LAST(clk, 18);
#ifdef BART_PHASE_CLOCKS
  if (clk >= 0 && poll_loads) atomicAdd((unsigned long long *)&clk_lds[clk][kClockPh - 1],
                                        (unsigned long long)poll_loads);
#endif
  lds_barrier();
  return nseg;
}

// Total of word k over all mailboxes: the segments summed in increasing order.
template <class SH>
__device__ __forceinline__ double seg_total(const SH &sh, int nseg, int K, int k) {
  double acc = 0.0;
  for (int seg = 0; seg < nseg; ++seg) acc += sh.part[seg * K + k];
  return acc;
}

// Grid-wide sum of one fp64 word per workgroup (sigma^2 step), into sh.tot[0].
template <class SH>
__device__ __forceinline__ void gather_total(const SweepArgs *__restrict__ A, SH &sh, int par,
                                             uint32_t seq, int nsum, uint32_t limit) {
  const int nseg = gather_polls(A, sh, par, seq, 1, nsum, limit);
  if (threadIdx.x == 0) sh.tot[0] = seg_total(sh, nseg, 1, 0);
  lds_barrier();
}

// Trace record of tree step j (written by the tree's owner): counts and
// partial sums per slot of the larger tree, new values of the final tree.
__device__ __noinline__ void trace_tree_step(bart_trace *R, Shared &sh, const Ctx &c, int j,
                                             int64_t s, int H) {
  const int t = threadIdx.x;
  const int eta = c.pr.eta;
  const int acc = sh.flags & 1, merged = (sh.flags >> 1) & 1;
  if (t < 256) {
    const int rnk = c.rank_of[t];
    const bool in = rnk < kNullRank && t < 2 * H;  // a leaf of the larger tree
    R->count[t] = in ? (int32_t)sh.cntd[rnk] : 0;
    R->sum[t] = in ? sh.S[rnk] : 0.0;
    float lv = 0.f;
    if (in && !(merged && (t >> 1) == eta)) lv = sh.newv[rnk];
    if (merged && t == eta) lv = sh.newv_m;
    R->leaf_new[t] = lv;
  }
  if (t == 0) {
    R->kind = 0;
    R->tree = j;
    R->sweep = s;
    R->move = c.pr.move;
    R->eta = eta;
    R->axis = c.pr.axis;
    R->cut = c.pr.cut;
    R->n_grow_cand = c.pr.nG;
    R->n_prune_cand = c.pr.nP;
    R->accept = acc;
    R->n_leaves = c.pr.L;
    R->log_r = sh.dec_logr;
    R->ln_u = c.pr.ln_u;
    R->log_r_scale = 0.0;
    R->ssr = 0.0;
    R->sigma2 = sh.sigma2;
  }
  if (t < 10) R->pad[t] = 0;
}

// Decision and leaf draws of one tree from the gathered per-segment partials
// (sh.part, nseg segments of K = L+1 words), the same in every workgroup.
// The MH decision (item 9) and every draw (items 4, 5, 10) are computed at
// once by different waves: the draws do not depend on the decision, only
// which of them is used.  Waves 0-3 handle the two leaves of the move (the
// decision, each child's own draw, the merged draw), waves 4-7 the other
// leaves; each wave sums the segments of the words it needs with the
// fixed-order DPP tree (nseg <= 32).  Writes sh.flags, dec_logr, and per
// rank cntd, S, newv and the final residual delta dlt, plus newv_m for a
// merged move.
// Move statistics of workgroup 0 (GROW proposed, PRUNE proposed, GROW
// accepted, PRUNE accepted, tree steps, leaves after the step) for the tree
// step whose proposal is c and whose decision flags are still in sh.flags.
// One thread; called where its wave would otherwise wait (the gather of the
// next tree step, the sigma^2 step, the end of the launch).
__device__ __forceinline__ void count_move(Shared &sh, const Ctx &c) {
  const int move = c.pr.move, L = c.pr.L;
  const int acc = sh.flags & 1, merged = (sh.flags >> 1) & 1;
  sh.stats[0] += move == kGrow;
  sh.stats[1] += move == kPrune;
  sh.stats[2] += move == kGrow && acc;
  sh.stats[3] += move == kPrune && acc;
  sh.stats[4] += 1;
  sh.stats[5] += (uint64_t)(L - merged);
}

// The parts of tree j's decision that need only counts (sec. 3.3 items 4,
// 5, 9, 10): for every leaf of known count (all but the children of a GROW)
// prec = n / s2 + 1 / v2 and the draw mean + z / sqrt(prec) written as
// S la + lb; the merged leaf of eta; for a PRUNE, the determinant term and
// the denominators of the likelihood ratio.  Before the gather, on wave 1
// when the tree is small (L + 5 <= 64 threads), else on waves 0-3: the
// polls run on the last waves.  The previous tree step's move statistics
// (its flags are still in sh.flags) are counted by thread 128 of workgroup 0.
__device__ __forceinline__ void pre_decide(const SweepArgs *__restrict__ A, Shared &sh,
                                           const Ctx &c, const TreeData &td, int uncounted) {
  const int L = c.pr.L;
  const int u0 = L + 5 <= 64 ? 64 : 0, nthreads = L + 5 <= 64 ? 64 : 256;
  if (uncounted >= 0 && threadIdx.x == 128) count_move(sh, sh.ctx[uncounted & (kRing - 1)]);
  const int u = (int)threadIdx.x - u0;
  if (u < 0 || u >= nthreads) return;
  const int move = c.pr.move, eta = c.pr.eta;
  const int kl = c.pr.rank_l, kr = c.pr.rank_r;
  const double s2 = sh.sigma2, v2 = A->sigma_mu * A->sigma_mu;
  // prec = n / s2 + 1 / v2 = e / (s2 v2) with e = s2 + n v2, so the draw
  // mean + z / sqrt(prec) is S v2 / e + mu_mu s2 / e + z sqrt(s2 v2 / e):
  // one division and one square root
  auto consts = [&](double n, double z, double &la, double &lb) {
    const double ie = 1.0 / (s2 + n * v2);
    la = v2 * ie;
    lb = A->mu_mu * s2 * ie + z * sqrt(s2 * v2 * ie);
  };
  if (u < L) {
    const int h = c.heap_of[u];
    const bool child = (move == kGrow) && ((h >> 1) == eta);
    if (!child) {
      const double n = (double)td.cnt[u];
      consts(n, td.z[u], sh.la[u], sh.lb[u]);
      sh.lnm[u] = n * (double)td.mu[u];
    }
  } else if (u == L && move != kNone) {
    const double n = move == kGrow ? (double)td.eta_cnt : (double)td.cnt[kl] + (double)td.cnt[kr];
    consts(n, td.eta_z, sh.ma, sh.mb);
  } else if (u >= L + 1 && u <= L + 4 && move == kPrune) {
    // one quantity per thread, so the divisions and the log run side by side
    const double nl = (double)td.cnt[kl], nr = (double)td.cnt[kr], np = nl + nr;
    const double eL = s2 + nl * v2, eR = s2 + nr * v2, eP = s2 + np * v2;
    if (u == L + 1)
      sh.pdL = 1.0 / eL;
    else if (u == L + 2)
      sh.pdR = 1.0 / eR;
    else if (u == L + 3)
      sh.pdP = 1.0 / eP;
    else
      sh.pdet = 0.5 * log(s2 * eP / (eL * eR));
  } else if (u == L + 1 && move == kGrow) {
    // the parent eta of a GROW keeps its count: its denominator is known
    const double eP = s2 + (double)td.eta_cnt * v2;
    sh.pdP = 1.0 / eP;
    sh.gs2eP = s2 * eP;
    sh.lgs2eP = log(s2 * eP);
  }
}

// 1/x from the hardware reciprocal and two Newton steps (within an ulp or two
// of the division; used where the sums have just arrived, on the critical
// path of the tree step).
__device__ __forceinline__ double rcp_fast(double x) {
  double r = __builtin_amdgcn_rcp(x);
  r = fma(fma(-x, r, 1.0), r, r);
  return fma(fma(-x, r, 1.0), r, r);
}

// ln x for a positive normal x to about 3e-7 absolute: the exponent exactly,
// the logarithm of the mantissa m in [0.5, 1) in fp32.
__device__ __forceinline__ double log_fast(double x) {
  const int e = __builtin_amdgcn_frexp_exp(x);
  const double m = __builtin_amdgcn_frexp_mant(x);
  return (double)e * 0.69314718055994530942 + (double)__logf((float)m);
}
// The accept decisions use log_fast only where it cannot change them: when
// ln u lies within this margin (times 1 + |ln x|) of the fast log r, the
// full fp64 logarithm decides, so every decision is the one fp64 takes.
constexpr double kLogFastMargin = 1e-5;

// Tree j's decision once the sums are in (sec. 3.3 items 8-10): wave 0 the
// MH ratio and accept, waves 1-2 the draws of the two move leaves (each
// takes the decision as well, so the residual delta it stores is final),
// wave 3 the merged draw, waves 4-7 every other leaf.  Every workgroup runs this on
// identical totals.
__device__ __forceinline__ void decide_step(const SweepArgs *__restrict__ A, Shared &sh,
                                            const Ctx &c, const TreeData &td, int nseg) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int move = c.pr.move, L = c.pr.L;
  const int kl = c.pr.rank_l, kr = c.pr.rank_r;
  const int K = L + 1;
  const double s2 = sh.sigma2, v2 = A->sigma_mu * A->sigma_mu;
  // this lane's segment partial of word k (0 past the segments); the read
  // index is clamped so every lane reads in bounds without a branch
  auto seg_part = [&](int k) {
    const double x = sh.part[(lane < nseg ? lane : 0) * K + k];
    return lane < nseg ? x : 0.0;
  };
  auto total = [&](int k) { return wave_total63(seg_part(k)); };  // valid in lane 63
  // conditional draw of a GROW child, whose count n comes with the sums:
  // with e = s2 + n v2, prec = e / (s2 v2), the mean is (S v2 + mu_mu s2) / e
  // and the sd sqrt(s2 v2 / e)
  // (the sd in fp32: its relative error, ~6e-8, is far below the leaf
  // tolerance)
  auto draw_child = [&](double e, double Sf, double z) {
    const double ie = rcp_fast(e);
    return (float)((Sf * v2 + A->mu_mu * s2) * ie + z * (double)sqrtf((float)(s2 * v2 * ie)));
  };
  if (move != kNone && wave < 4) {
    // everything this part reads from LDS besides the sums, read up front
    const double eta_cnt = (double)td.eta_cnt;
    const float eta_mu = td.eta_mu, mul = td.mu[kl], mur = td.mu[kr];
    const double cl = (double)td.cnt[kl], cr = (double)td.cnt[kr];
    const double lnml = sh.lnm[kl], lnmr = sh.lnm[kr];
    const double lal = sh.la[kl], lar = sh.la[kr], lbl = sh.lb[kl], lbr = sh.lb[kr];
    const double zl = td.z[kl], zr = td.z[kr];
    const double ma = sh.ma, mb = sh.mb, pdP = sh.pdP;
    const double pdet = sh.pdet, pdL = sh.pdL, pdR = sh.pdR, gs2eP = sh.gs2eP;
    const double lgs2eP = sh.lgs2eP;
    const double c_prior = c.pr.c_prior, ln_u = c.pr.ln_u;
    double nR = move == kGrow ? seg_part(L) : 0.0, Rl = seg_part(kl), Rr = seg_part(kr);
    wave_totals3(nR, Rl, Rr);
    if (lane == 63) {
      // counts and partial sums S_h = R_h + n_h (old value) of the two leaves
      const bool grow = move == kGrow;
      const double nl = grow ? eta_cnt - nR : cl, nr = grow ? nR : cr;
      const float mol = grow ? eta_mu : mul, mor = grow ? eta_mu : mur;
      const double Sl = grow ? Rl + nl * (double)mol : Rl + lnml;
      const double Sr = grow ? Rr + nr * (double)mor : Rr + lnmr;
      const double mm = A->mu_mu;
      const double tL = Sl - nl * mm, tR = Sr - nr * mm, tP = (Sl + Sr) - (nl + nr) * mm;
      // log r: the log marginal-likelihood ratio of splitting a leaf into
      // (L, R) -- the partial residuals of a leaf with n points, its
      // N(mu_mu, v2) value integrated out (sec. 2.1), are N(mu_mu 1,
      // s2 I + v2 1 1^T), so LLR = 1/2 ln(s2 eP / (eL eR)) + v2 / (2 s2)
      // (tL^2/eL + tR^2/eR - tP^2/eP) with e = s2 + n v2 and t = S - n mu_mu,
      // the count-only parts from pre_decide -- plus the count-free terms
      // (GROW: ln(s2 eP) from pre_decide minus a fast ln(eL eR), redone in
      // full fp64 when ln u falls within kLogFastMargin of the result)
      auto log_r = [&]() {
        if (grow) {
          const double eL = s2 + nl * v2, eR = s2 + nr * v2;
          const double p = eL * eR, r = rcp_fast(p);
          const double q = v2 / (2.0 * s2) * (tL * tL * (eR * r) + tR * tR * (eL * r) - tP * tP * pdP);
          const double lp = log_fast(p);
          const double fast = c_prior + (0.5 * (lgs2eP - lp) + q);
          if (fabs(ln_u - fast) > kLogFastMargin * (1.0 + fabs(lp))) return fast;
          return c_prior + (0.5 * log(gs2eP * r) + q);
        }
        const double llr = pdet + v2 / (2.0 * s2) * (tL * tL * pdL + tR * tR * pdR - tP * tP * pdP);
        return c_prior - llr;
      };
      const float vm = (float)((Sl + Sr) * ma + mb);
      if (wave == 0) {
        const double logr = log_r();
        const int acc = ln_u < logr ? 1 : 0;
        const int merged = (grow && !acc) || (move == kPrune && acc);
        sh.dec_logr = logr;
        sh.flags = acc | (merged << 1);
      } else if (wave == 3) {
        sh.newv_m = vm;
      } else {
        // the two leaves of the move: each of waves 1 and 2 takes the
        // decision too (the same arithmetic on the same totals as wave 0),
        // so its residual delta is final: the child's own draw, or the
        // merged value of eta
        const bool left = wave == 1;
        const int k = left ? kl : kr;
        const double Sk = left ? Sl : Sr, nk = left ? nl : nr;
        const float mo = left ? mol : mor;
        const float v = grow ? draw_child(s2 + nk * v2, Sk, left ? zl : zr)
                             : (float)(Sk * (left ? lal : lar) + (left ? lbl : lbr));
        const int acc = ln_u < log_r() ? 1 : 0;
        const int merged = (grow && !acc) || (move == kPrune && acc);
        sh.cntd[k] = nk;
        sh.S[k] = Sk;
        sh.newv[k] = v;
        sh.dlt[k] = merged ? mo - vm : mo - v;
      }
    }
  }
  if (move == kNone && t == 0) {
    sh.dec_logr = 0.0;
    sh.flags = 0;
  }
  const int first = move != kNone ? wave - 4 : wave, stride = move != kNone ? 4 : kWaves;
  for (int k = first < 0 ? L : first; k < L; k += stride) {
    if (move != kNone && (k == kl || k == kr)) continue;
    const double R = total(k);
    if (lane == 63) {
      const double Sk = R + sh.lnm[k];
      const float v = (float)(Sk * sh.la[k] + sh.lb[k]);
      sh.cntd[k] = (double)td.cnt[k];
      sh.S[k] = Sk;
      sh.newv[k] = v;
      sh.dlt[k] = td.mu[k] - v;
    }
  }
}

// After the decision of tree j: its owner workgroup (j mod G) stores the
// final tree (values and counts of its leaves, structure change) and the
// trace record.
__device__ __forceinline__ void finish_tree(const SweepArgs *__restrict__ A, const Launch &Lc,
                                            Shared &sh, const Ctx &c, int j, int64_t s,
                                            int step) {
  const int t = threadIdx.x, w = wg_id(A), G = A->G, H = A->H;
  const int move = c.pr.move, eta = c.pr.eta, L = c.pr.L;
  const int kl = c.pr.rank_l, kr = c.pr.rank_r;
  const int acc = sh.flags & 1, merged = (sh.flags >> 1) & 1;
  const float vm = sh.newv_m;
  // the owner stores the final tree: values and counts of its leaves,
  // structure change, move statistics and the trace record
  if (j % G == w) {
    if (t < L) {
      const int h = c.heap_of[t];
      const bool to_eta = merged && (t == kl || t == kr);
      const int f = to_eta ? eta : h;
      const double nf = to_eta ? sh.cntd[kl] + sh.cntd[kr] : sh.cntd[t];
      gbl(A->leaf)[(int64_t)j * 2 * H + f] = to_eta ? vm : sh.newv[t];
      gbl(A->count)[(int64_t)j * 2 * H + f] = (int32_t)nf;
    }
    if (t == 0) {
      const gptr<uint8_t> ct = gbl(A->cut) + (int64_t)j * H;
      const gptr<uint16_t> ax = gbl(A->axis) + (int64_t)j * H;
      if (move == kGrow && acc) {
        ax[eta] = (uint16_t)c.pr.axis;
        ct[eta] = (uint8_t)c.pr.cut;
        if (2 * eta < H) ct[2 * eta] = 0;
        if (2 * eta + 1 < H) ct[2 * eta + 1] = 0;
      }
      if (move == kPrune && acc) ct[eta] = 0;
    }
    if (Lc.trace) trace_tree_step(Lc.trace + step, sh, c, j, s, H);
  }
}


// The sigma^2 step after this workgroup's per-wave sums of squared
// residuals are in sh.wave_part: the next sweep's proposals (owners) and
// normals, the grid-wide SSR in a fixed order, and the draw, made by every
// workgroup alike.
template <class SH>
__device__ __forceinline__ void sigma2_tail(const SweepArgs *__restrict__ A, const Launch &Lc,
                                            SH &sh, int64_t s, int step, uint32_t seq,
                                            int par) {
  const int t = threadIdx.x, w = wg_id(A), m = A->m;
  const uint64_t seed = Lc.seed;
  const bool tracing = Lc.trace != nullptr;
  // the gamma variate of this sweep's sigma^2 draw, on the last wave (one
  // that owns no tree unless a workgroup owns more than 7), while the
  // others propose
  if (!A->probit && t == kBlock - 64) sh.sig_gamma = sigma2_gamma(A, seed, s);
  // the next sweep's proposals (owners) and normals, published by the
  // release below together with this sweep's tree writes
  BART_SCLOCK(1);
  gen_proposals(A, seed, s + 1, 0);
  BART_SCLOCK(2);
  gen_normals(A, seed, s + 1, 0);
  BART_SCLOCK(3);
  __syncthreads();
  BART_SCLOCK(4);
  if (t < 64) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");  // publish_workgroup, stamped
  BART_SCLOCK(5);
  if (t == 0) {
    double acc = 0.0;
    for (int u = 0; u < kWaves; ++u) acc += sh.wave_part[u];
    post(A, sh, par, 0, mk_word(seq, pack_f64(acc)));
  }
  gather_total(A, sh, par, seq, 1, Lc.spin_limit);
  BART_SCLOCK(6);
  // acquire by the wave that polled (a one-word gather polls on the last
  // wave); the other waves read what it publishes after the barrier at the
  // end of this step, and until then only LDS
  if (t >= kBlock - 64) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  if (t == 0) {
    const double ssr_all = sh.tot[0];
    // the probit model holds sigma^2 at 1 and draws latents instead
    const double s2 = A->probit ? sh.sigma2 : sigma2_of(A, ssr_all, sh.sig_gamma);
    sh.sigma2 = s2;
    if (w == 0) {
      A->ctl->sigma2 = s2;
      A->ctl->sweep = s + 1;
      if (tracing) {
        bart_trace *R = Lc.trace + step;
        R->kind = 1;
        R->tree = m;
        R->sweep = s;
        R->move = 0;
        R->ssr = ssr_all;
        R->sigma2 = s2;
      }
    }
  }
  if (tracing && w == 0) {
    // the rest of the sigma^2 record is zero
    bart_trace *R = Lc.trace + step;
    if (t < 256) {
      R->count[t] = 0;
      R->sum[t] = 0.0;
      R->leaf_new[t] = 0.f;
    }
    if (t >= 1 && t < 10) R->pad[t] = 0;
    if (t == 1) {
      R->eta = R->axis = R->cut = R->n_grow_cand = R->n_prune_cand = R->accept = 0;
      R->n_leaves = 0;
      R->log_r = R->ln_u = R->log_r_scale = 0.0;
      R->pad[0] = 0;
    }
  }
  __syncthreads();
}

template <int V, int IB>
__device__ __forceinline__ void sweep_body(const SweepArgs *__restrict__ A, const Launch &Lc,
                                           Shared &sh) {
  using IC = IdxChunk<IB>;
  using ChunkT = typename IC::T;
  // the thread index is re-read opaquely at every step (see the loop), so
  // addresses derived from it are recomputed rather than kept in registers
  // (or spilled) across the whole loop
  int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int w = wg_id(A);
  const int G = A->G, H = A->H, m = A->m;
  const uint64_t seed = Lc.seed;
  const bool tracing = Lc.trace != nullptr;

  float r[V][4];
  uint32_t rk[V];   // ranks of the tree being decided, 4 x 8 bits per chunk
  uint32_t rk2[V];  // ranks of the next tree
  ChunkT rawc[V];
  uint32_t rawx[V];
  // chunk v of this thread exists iff t + v kBlock < lim, lim uniform over
  // the workgroup: no per-chunk mask is kept across the loop (a chunk past
  // the end has no load of its own and routes to the null rank)
  const int32_t lim = A->chunks - w * V * kBlock;
  auto chunk_ok = [&](int v) { return t + v * kBlock < lim; };
  // bit b: observation 4 chunk + b exists (sigma^2 step and epilogue)
  auto ok4 = [&](int v) -> uint32_t {
    const int32_t rem = A->n - 4 * ((w * V + v) * kBlock + t);
    return !chunk_ok(v) ? 0u : (rem >= 4 ? 15u : ((1u << rem) - 1u));
  };
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const int32_t ch = (w * V + v) * kBlock + t;
    r[v][0] = r[v][1] = r[v][2] = r[v][3] = 0.f;
    if (chunk_ok(v)) {
      const gptr<const float> q = gbl((const float *)A->resid) + 4 * (int64_t)ch;
      r[v][0] = q[0];
      r[v][1] = q[1];
      r[v][2] = q[2];
      r[v][3] = q[3];
    }
    rk[v] = rk2[v] = 0;
    rawc[v] = 0;
    rawx[v] = 0;
  }
  for (int k = t; k < kBinFloats; k += kBlock) sh.bins[k] = 0.f;
  if (t == 0) {
    sh.abort_flag = 0;
    sh.dev_err = 0;
    sh.nr[0] = sh.nr[1] = 0;
    sh.sigma2 = A->ctl->sigma2;
  }
  // ranks from kNullRank on: zero delta, slot 0
  if (t >= kNullRank && t < 256) sh.dlt[t] = 0.f;
  for (int q = t; q < kRing * (256 - kNullRank); q += kBlock)
    sh.ctx[q / (256 - kNullRank)].heap_of[kNullRank + q % (256 - kNullRank)] = 0;
  if (t < 6) sh.stats[t] = 0;
  int uncounted = -1;  // tree step whose move statistics workgroup 0 has yet to count
  int clk = -1;        // phase-clock slot of the current step (diagnostic build)

  // ---- helpers over the pipeline ----
  // issue the index-row and predictor-row loads of tree `tree` (its proposal in ctx)
  auto issue_rows = [&](int tree) {
    const Ctx &c = sh.ctx[tree & (kRing - 1)];
    const gptr<const ChunkT> row =
        gbl((const ChunkT *)((const char *)A->idx + (int64_t)tree * A->ldi * IB));
    const gptr<const uint32_t> xrow = gbl((const uint32_t *)(A->X + (int64_t)c.pr.axis * A->ldx));
    // unconditional loads (chunk 0 stands in for a chunk past the end)
#pragma unroll
    for (int v = 0; v < V; ++v) {
      const int32_t ch = (w * V + v) * kBlock + t;
      const int32_t cc = chunk_ok(v) ? ch : 0;
      rawc[v] = row[cc];
      rawx[v] = xrow[cc];
    }
  };
  // route this workgroup's points through tree `tree` (rows already loaded):
  // rank of each point's leaf in the larger tree, GROW right-count into nr
  auto route = [&](int tree, uint32_t (&out)[V]) {
    const Ctx &c = sh.ctx[tree & (kRing - 1)];
    const int move = c.pr.move, eta = c.pr.eta, cutv = c.pr.cut;
    const int grow_eta = move == kGrow ? eta : -1;
    // leaf of every point in the larger tree, then all rank lookups at once
    int cp[V][4];
    int nr = 0;
    if (grow_eta >= 0) {
#pragma unroll
      for (int v = 0; v < V; ++v) {
        // a chunk past the end: index 0, the null rank, for all its points
        const ChunkT rc = chunk_ok(v) ? rawc[v] : (ChunkT)0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int ci = IC::get(rc, b);
          const int xi = (rawx[v] >> (8 * b)) & 0xff;
          const bool in = ci == grow_eta;
          const int right = xi >= cutv;
          cp[v][b] = in ? 2 * eta + right : ci;  // below 256: eta < 128
          nr += __popcll(__ballot(in && right));  // wave-uniform
        }
      }
    } else {
      // not a GROW (a uniform branch): every point keeps its leaf, and the
      // predictor bytes, loaded all the same, go unused
#pragma unroll
      for (int v = 0; v < V; ++v) {
        const ChunkT rc = chunk_ok(v) ? rawc[v] : (ChunkT)0;
#pragma unroll
        for (int b = 0; b < 4; ++b) cp[v][b] = IC::get(rc, b);
      }
    }
    int r0[V][4];
#pragma unroll
    for (int v = 0; v < V; ++v)
#pragma unroll
      for (int b = 0; b < 4; ++b) r0[v][b] = c.rank_of[cp[v][b]];
    // slot 0 marks a padding point (its index entry, or no load at all past
    // the last chunk) and has the null rank, whose delta is 0 and which falls
    // in no bin, so no per-point mask is needed; any other non-leaf slot is
    // an inconsistent cache, rank kBadRank (no bin, zero delta), flagged
    int worst = 0;
#pragma unroll
    for (int v = 0; v < V; ++v) {
      uint32_t pk = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        worst = max(worst, r0[v][b]);
        pk |= (uint32_t)r0[v][b] << (8 * b);
      }
      out[v] = pk;
    }
    if (worst == kBadRank) sh.dev_err = 1;
    if (lane == 0 && nr) atomicAdd(&sh.nr[tree & 1], nr);
  };
  // partial sums of tree `tree` from the current residuals: per-lane private
  // LDS bins in kSets sets per lane (with two, the points of chunk positions
  // 0, 2 go to set 0, those of 1, 3 to set 1; with four, position e to set
  // e), so each lane runs kSets independent chains of read-modify-writes,
  // for up to kRegRanks ranks at a time (a plain read-modify-write: LDS float
  // atomics are many times slower; ranks outside the pass, the null rank of
  // padding points among them, add 0 to a bin of the pass, so there is no
  // branch per point); then a fixed-order fp64 reduction of the kSets x 8
  // bins of each lane position and a DPP tree over the lanes; larger trees
  // take several passes.  The wave that forms the total
  // of rank k posts it as word k of this workgroup's mailbox for the step
  // that decides the tree (buffer par, step number seq), and after the first
  // bin barrier thread kBlock-1 posts the GROW right-count that route(tree)
  // gathered as word L: no barrier stands between the totals and the post
  // (only between passes).
  // four sets with 8 chunks per thread (chains of 8 read-modify-writes
  // rather than 16: four chains 2547 -> 2562 chain-sweeps/s)
  constexpr int kSets = V >= 8 ? 4 : 2;
  constexpr int kRegRanks = kBinFloats / (kSets * kBlock);  // 32 or 16
  static_assert(kMaxLeaves % kRegRanks == 0 && kNullRank / kRegRanks >= kMaxLeaves / kRegRanks,
                "the null rank must fall outside every bin pass");
  auto reduce = [&](int tree, const uint32_t (&rks)[V], int par, uint32_t seq) {
    const int L = sh.ctx[tree & (kRing - 1)].pr.L;
    const int wl = wave * 64 + lane;
    for (int base = 0; base < L; base += kRegRanks) {
      // the bin of rank k is k mod kRegRanks; a point outside the pass adds
      // 0 to its bin there (exact: a bin never holds -0).  Bins of different
      // sets never share an address, so a pair (one point of each set) is
      // read together and written together
#pragma unroll
      for (int v = 0; v < V; ++v)
#pragma unroll
        for (int b0 = 0; b0 < 4; b0 += kSets) {
          const uint32_t pass = (uint32_t)(base / kRegRanks);
          int q[kSets];
          float x[kSets], cur[kSets];
#pragma unroll
          for (int e = 0; e < kSets; ++e) {
            const uint32_t rr = (rks[v] >> (8 * (b0 + e))) & 0xffu;
            q[e] = ((int)(rr % kRegRanks) * kSets + e) * kBlock + wl;
            x[e] = rr / kRegRanks == pass ? r[v][b0 + e] : 0.f;
          }
#pragma unroll
          for (int e = 0; e < kSets; ++e) cur[e] = sh.bins[q[e]];
#pragma unroll
          for (int e = 0; e < kSets; ++e) sh.bins[q[e]] = cur[e] + x[e];
        }
      if (base == 0) BART_CLOCK(clk, 9);
      lds_barrier();
      if (base == 0) BART_CLOCK(clk, 10);
      if (base == 0 && t == kBlock - 1) {
        // cleared for route(tree + 2), the next to count into this slot
        post(A, sh, par, L, mk_word(seq, (uint64_t)sh.nr[tree & 1]));
        sh.nr[tree & 1] = 0;
      }
      for (int k = base + wave; k < min(L, base + kRegRanks); k += kWaves) {
        // the kSets x 8 bins of this lane position (sets x waves): all read,
        // then cleared, then summed in a fixed tree
        double x[kSets * kWaves];
#pragma unroll
        for (int q = 0; q < kSets * kWaves; ++q)
          x[q] = (double)sh.bins[(((k - base) * kSets + q / kWaves) * kWaves + q % kWaves) * 64 + lane];
#pragma unroll
        for (int q = 0; q < kSets * kWaves; ++q)
          sh.bins[(((k - base) * kSets + q / kWaves) * kWaves + q % kWaves) * 64 + lane] = 0.f;
#pragma unroll
        for (int w2 = 1; w2 < kSets * kWaves; w2 *= 2)
#pragma unroll
          for (int q = 0; q < kSets * kWaves; q += 2 * w2) x[q] += x[q + w2];
        const double tot = wave_total63(x[0]);
        if (lane == 63) post(A, sh, par, k, mk_word(seq, pack_f64(tot)));
        if (k == 0) BART_CLOCK(clk, 11);
      }
      if (base + kRegRanks < L) lds_barrier();
    }
  };
  // proposals of trees j0.. j0+2 into the ring, rank tables, rows of j0,
  // route of j0, rows of j0+1, decision data of j0, partial sums of j0
  // (posted for launch step `next`, which decides tree j0)
  auto refill = [&](int j0, int64_t s, int next) {
    for (int q = 0; q < 3; ++q)
      if (j0 + q < m) {
        const uint32_t wd = load_prop_word(A, j0 + q);
        if (t < kPropWords) ((uint32_t *)&sh.ctx[(j0 + q) & (kRing - 1)].pr)[t] = wd;
      }
    lds_barrier();
    for (int q = 0; q < 3; ++q)
      if (j0 + q < m) build_ranks(A, sh.ctx[(j0 + q) & (kRing - 1)]);
    lds_barrier();
    issue_rows(j0);
    const TdRegs tr0 = load_tree_data(A, sh.ctx[j0 & (kRing - 1)], j0, s);
    route(j0, rk);
    if (j0 + 1 < m) issue_rows(j0 + 1);
    store_tree_data(sh.td[j0 & 1], sh.ctx[j0 & (kRing - 1)], tr0);
    wait_vm_loads();  // the rows of j0 + 1 are in before the posts
    reduce(j0, rk, next & 1, (uint32_t)next + 2);
  };

  // ---- prologue: proposals and normals of the first sweep, grid rendezvous
  int64_t s = Lc.s0;
  int j = Lc.j0;
  if (j < m) {
    gen_proposals(A, seed, s, j);
    gen_normals(A, seed, s, j);
  }
  publish_workgroup();
  if (t == 0) post(A, sh, 1, 0, mk_word(1, 0));
  gather_total(A, sh, 1, 1, 0, Lc.spin_limit);
  // acquire by the wave that polled (a one-word gather polls on the last
  // wave); the barrier orders the other waves after it
  if (t >= kBlock - 64) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  __syncthreads();
  if (j < m && !sh.abort_flag) refill(j, s, 0);

#pragma unroll 1
  for (int step = 0; step < Lc.n_steps; ++step) {
    if (sh.abort_flag) break;
    asm volatile("" : "+v"(t));
    lane = t & 63;
    wave = t >> 6;
    const uint32_t seq = (uint32_t)step + 2;
    const int par = step & 1;
    if (j < m) {
      // ================= tree step j =================
      Ctx &c = sh.ctx[j & (kRing - 1)];
      const int move = c.pr.move, eta = c.pr.eta, L = c.pr.L;
      const int kl = c.pr.rank_l, kr = c.pr.rank_r;
      const bool more1 = (j + 1 < m) && (step + 1 < Lc.n_steps);  // tree j+1 follows
      const bool more2 = more1 && (j + 2 < m);
      const bool more3 = more2 && (j + 3 < m);
      // 1. route tree j+1 (its rows were loaded a step ago); this
      //    workgroup's partial sums of tree j and its GROW right-count were
      //    posted by the reduce that formed them
      clk = clock_slot(step);
      BART_CLOCK(clk, 0);
      BART_CLOCK_LAST(clk, 13);
      if (more1) route(j + 1, rk2);
      BART_CLOCK(clk, 1);
      BART_CLOCK_LAST(clk, 14);
      // 2. while the mailboxes fill: load rows of j+2, the decision data of
      //    j+1 and the proposal of j+3
      // (the small loads first: nothing waits behind the row loads)
      const int j1 = more1 ? j + 1 : j, j3 = more3 ? j + 3 : j;
      const TdRegs tdn = load_tree_data(A, sh.ctx[j1 & (kRing - 1)], j1, s);
      const uint32_t pw3 = load_prop_word(A, j3);
      BART_CLOCK_LAST(clk, 15);
      if (more2) issue_rows(j + 2);
      BART_CLOCK_LAST(clk, 16);
      // 3. totals of tree j, in the same order in every workgroup: polls into
      //    per-segment partials, then one wave reduces a word over the
      //    segments with the fixed-order DPP tree (nseg <= 32 lanes).  The
      //    polls run on the last waves; before the gather, wave 3 builds the
      //    rank table of tree j+2 (its proposal was staged a step ago; 4
      //    slots per lane) and wave 1 (waves 0-3 for large trees) computes
      //    tree j's count-only constants
      const int K = L + 1;
      if (more2 && wave == 3)
#pragma unroll
        for (int i = 0; i < 4; ++i) build_rank_slot(A, sh.ctx[(j + 2) & (kRing - 1)], 64 * i + lane);
      pre_decide(A, sh, c, sh.td[j & 1], w == 0 ? uncounted : -1);
      BART_CLOCK(clk, 2);
      const int nseg = gather_polls(A, sh, par, seq, K, L, Lc.spin_limit, clk);
      BART_CLOCK(clk, 3);
      decide_step(A, sh, c, sh.td[j & 1], nseg);
      BART_CLOCK(clk, 4);
      // stage what later trees need
      if (more3 && t < kPropWords) ((uint32_t *)&sh.ctx[(j + 3) & (kRing - 1)].pr)[t] = pw3;
      if (more1) store_tree_data(sh.td[(j + 1) & 1], sh.ctx[(j + 1) & (kRing - 1)], tdn);
      lds_barrier();
      BART_CLOCK(clk, 5);
      wait_vm_loads();  // the rows of j+2 are in before this step's stores
      // 4. residuals and index row (item 11): the delta of every rank is
      //    final (a point in a child of eta of a merged move takes the
      //    merged value); such a point also takes the index eta
      const int flags = sh.flags, acc = flags & 1, merged = (flags >> 1) & 1;
      const bool changed = acc && move != kNone;
      const gptr<ChunkT> row = gbl((ChunkT *)((char *)A->idx + (int64_t)j * A->ldi * IB));
      float dl[V][4];
#pragma unroll
      for (int v = 0; v < V; ++v)
#pragma unroll
        for (int b = 0; b < 4; ++b) dl[v][b] = sh.dlt[(rk[v] >> (8 * b)) & 0xff];
#pragma unroll
      for (int v = 0; v < V; ++v)
#pragma unroll
        for (int b = 0; b < 4; ++b) r[v][b] += dl[v][b];
      if (changed) {
#pragma unroll
        for (int v = 0; v < V; ++v) {
          bool touch = false;
          ChunkT out = 0;
          // every rank's heap slot read unconditionally (no exec mask per
          // point; ranks from kNullRank on have slot 0), then selected
          int hs[4];
#pragma unroll
          for (int b = 0; b < 4; ++b) hs[b] = c.heap_of[(rk[v] >> (8 * b)) & 0xff];
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int rnk = (rk[v] >> (8 * b)) & 0xff;
            const bool pair = (rnk == kl) || (rnk == kr);
            touch |= pair;
            out = IC::put(out, b, (merged && pair) ? eta : hs[b]);
          }
          // only an existing chunk has a point of the move's pair
          if (touch) row[(w * V + v) * kBlock + t] = out;
        }
      }
      BART_CLOCK(clk, 6);
      finish_tree(A, Lc, sh, c, j, s, step);
      uncounted = j;
      BART_CLOCK(clk, 7);
      // 5. tree j+1: partial sums from the updated residuals
      if (more1) {
        reduce(j + 1, rk2, (step + 1) & 1, (uint32_t)step + 3);
#pragma unroll
        for (int v = 0; v < V; ++v) rk[v] = rk2[v];
      } else {
        lds_barrier();
      }
      BART_CLOCK(clk, 8);
      BART_CLOCK_LAST(clk, 12);
      ++j;
    } else {
      // ================= sigma^2 step (sec. 3.3, "Sampling the error variance")
      clk = -1;
      BART_SCLOCK(0);
      if (w == 0 && t == kBlock - 1 && uncounted >= 0)
        count_move(sh, sh.ctx[uncounted & (kRing - 1)]);
      uncounted = -1;
      __syncthreads();  // this workgroup's tree writes are visible to all its threads
      double ssr = 0.0;
#pragma unroll
      for (int v = 0; v < V; ++v)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const double x = (double)r[v][b];  // 0 at padding points
          ssr += x * x;
        }
      ssr = wave_total63(ssr);
      if (lane == 63) sh.wave_part[wave] = ssr;
      sigma2_tail(A, Lc, sh, s, step, seq, par);
      if (A->probit)
#pragma unroll
        for (int v = 0; v < V; ++v)
          if (const uint32_t ok = ok4(v)) latent_chunk(A, seed, s, (w * V + v) * kBlock + t, ok, r[v]);
      j = 0;
      ++s;
      BART_SCLOCK(7);
      if (step + 1 < Lc.n_steps && !sh.abort_flag) refill(0, s, step + 1);
      BART_SCLOCK(8);
    }
  }

  // ---- epilogue: residuals back to HBM, statistics, device errors
#pragma unroll
  for (int v = 0; v < V; ++v)
    if (chunk_ok(v)) {
      const int32_t ch = (w * V + v) * kBlock + t;
      const gptr<float> q = gbl(A->resid) + 4 * (int64_t)ch;
      q[0] = r[v][0];
      q[1] = r[v][1];
      q[2] = r[v][2];
      q[3] = r[v][3];
    }
  if (w == 0 && t == kBlock - 1 && uncounted >= 0)
    count_move(sh, sh.ctx[uncounted & (kRing - 1)]);
  __syncthreads();
  if (w == 0 && t < 6) A->ctl->stats[t] += sh.stats[t];
  if (t == 0 && (sh.abort_flag || sh.dev_err))
    atomicOr(&A->ctl->error, (sh.abort_flag ? BART_DEVERR_TIMEOUT : 0u) |
                                 (sh.dev_err ? BART_DEVERR_CACHE : 0u));
}

template <int V, int IB>
__global__ void __launch_bounds__(kBlock) sweep_kernel(const SweepArgs *__restrict__ A, Launch Lc) {
  __shared__ Shared sh;
  // a workgroup left out (bart_debug_stall): every wait on it times out
  if ((int)blockIdx.x == Lc.absent_wg) return;
#ifdef BART_PHASE_CLOCKS
  for (int q = threadIdx.x; q < kClockSteps * kClockPh; q += kBlock)
    clk_lds[q / kClockPh][q % kClockPh] = 0;
  __syncthreads();
#endif
  const int c = (int)blockIdx.x / A->G;
  if (Lc.trace) Lc.trace += c * Lc.trace_stride;
  sweep_body<V, IB>(A + c, Lc, sh);
#ifdef BART_PHASE_CLOCKS
  __syncthreads();
  for (int q = threadIdx.x; q < kClockSteps * kClockPh; q += kBlock)
    g_phase_clock[blockIdx.x][q / kClockPh][q % kClockPh] = clk_lds[q / kClockPh][q % kClockPh];
#endif
}

// ------------------------------------------------------------------ streamed
// Residual cache in HBM (sec. 3.3 "Residuals cache"), for problems whose
// residuals do not fit in the registers of the grid.  The step structure and
// the grid protocol are those of sweep_body; the difference is the data
// pass: per tree step j one pass over this workgroup's points reads each
// residual once, adds tree j's delta (its route recomputed from the index
// row and predictor row), writes it back, rewrites the index row where the
// tree changed, and accumulates tree j+1's partial sums from the updated
// value (route of j+1 from its rows).  Partial sums are fp64 per lane.
// With ST (the chunks of a thread fit the stash, kStashCpt), the ranks of tree
// j+1 that this pass computes stay in LDS, one byte per point, for the pass
// of step j+1 that applies the tree: that pass then reads neither the index
// row nor the predictor row again (nor, without an index cache, a rolling
// row of leaves), and trees with more leaves than one bin pass holds take
// their extra passes from the stash too.  The LDS left after the bins and the
// stash holds the residuals of each thread's first chunks for the launch
// (resid_lds_chunks), so only the other chunks' residuals cross HBM every
// step.
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int IB, bool CF, bool ST>
__device__ __forceinline__ void sweep_body_stream(const SweepArgs *__restrict__ A, const Launch &Lc,
                                                  Shared &sh) {
  using IC = IdxChunk<IB>;
  using ChunkT = typename IC::T;
  // chunks of 4 points per batch (three batches in flight): without an index
  // cache two, so that the level-by-level predictor gathers of Algorithm 1
  // have twice the points in flight (one chunk: 374, two: 409 sweeps/s at
  // n = 1e6; four spill); with the rank stash also two, as its batches load
  // no rows of the tree they apply and would otherwise keep fewer bytes in
  // flight (n = 1e7: one chunk 183, two 194, three 180 sweeps/s)
  constexpr int U = (CF || ST) ? 2 : 1;
  constexpr int kPassRanks = ST ? kStashRanks : kSlotRanks;
  constexpr int kPos = ST ? kStashPos : 4;  // bins per lane and rank: chunk positions
  constexpr uint32_t kNull4 = kNullRank * 0x01010101u;  // a chunk of padding points
  uint32_t *const stash = (uint32_t *)(sh.bins + kStashOffset);  // [cpt][kBlock]
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, w = wg_id(A);
  const int m = A->m, cpt = A->cpt;
  const uint64_t seed = Lc.seed;
  // with the stash, the residuals of this thread's chunks 0..rc-1 stay in
  // LDS for the launch ([rc][kBlock] chunks after the stash; only this thread
  // touches its own), read from HBM here and written back at the end
  const int rc = ST ? resid_lds_chunks(cpt) : 0;
  f32x4 *const rcache = (f32x4 *)(sh.bins + kStashOffset + cpt * kBlock);
  for (int k = t; k < (ST ? kStashOffset + cpt * kBlock : kBinFloats); k += kBlock) sh.bins[k] = 0.f;
  for (int i = 0; i < rc; ++i) {
    const int32_t ch = (w * cpt + i) * kBlock + t;
    rcache[i * kBlock + t] =
        ch < A->chunks ? gbl((const f32x4 *)A->resid)[ch] : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  if (t == 0) {
    sh.abort_flag = 0;
    sh.dev_err = 0;
    sh.nr[0] = sh.nr[1] = 0;
    sh.sigma2 = A->ctl->sigma2;
  }
  // ranks from kNullRank on: zero delta, slot 0
  if (t >= kNullRank && t < 256) sh.dlt[t] = 0.f;
  for (int q = t; q < kRing * (256 - kNullRank); q += kBlock)
    sh.ctx[q / (256 - kNullRank)].heap_of[kNullRank + q % (256 - kNullRank)] = 0;
  if (t < 6) sh.stats[t] = 0;
  int uncounted = -1;  // tree step whose move statistics workgroup 0 has yet to count

  // leaf ranks in tree c's larger tree of the 4 points of a chunk.  Index 0
  // marks a padding point (its entry in the row, or a chunk past the end
  // whose loaded values were zeroed): the null rank, whose delta is 0 and
  // which falls in no bin; any other non-leaf slot is an inconsistent cache,
  // rank kBadRank (likewise inert), and bad keeps the largest rank seen so
  // the pass can flag it.
  // (grow_eta: eta of a GROW, -1 otherwise; eta and cut of the proposal,
  // read once per pass by the caller.  Without the rank stash, the GROW
  // right-count into *nrb when given: a ballot per point, which there keeps
  // fewer registers live than the packed-byte count of the stash kernels)
  auto ranks4 = [&](const Ctx &c, int grow_eta, int eta, int cutv, ChunkT rc, uint32_t rx,
                    uint32_t &bad, int *nrb) -> uint32_t {
    uint32_t pk = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int ci = IC::get(rc, b);
      const int xi = (rx >> (8 * b)) & 0xff;
      const bool in = ci == grow_eta;
      const int right = xi >= cutv;
      const int r0 = c.rank_of[in ? 2 * eta + right : ci];  // slot below 256: eta < 128
      if (!ST && nrb) *nrb += __popcll(__ballot(in && right));  // wave-uniform
      bad = max(bad, (uint32_t)r0);
      pk |= (uint32_t)r0 << (8 * b);
    }
    return pk;
  };
  // the same when the move is not a GROW: every point keeps its leaf
  auto ranks4_plain = [&](const Ctx &c, ChunkT rc, uint32_t &bad) -> uint32_t {
    uint32_t pk = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int r0 = c.rank_of[IC::get(rc, b)];
      bad = max(bad, (uint32_t)r0);
      pk |= (uint32_t)r0 << (8 * b);
    }
    return pk;
  };
  // the number of bytes of x that are zero (no carry crosses a byte)
  auto zero_bytes = [](uint32_t x) -> int {
    const uint32_t y = (x & 0x7f7f7f7fu) + 0x7f7f7f7fu;
    return __popc(~(y | x) & 0x80808080u);
  };

  // one pass: apply tree ja (-1: none), accumulate the ranks [lo, lo +
  // kPassRanks) of tree jn (-1: none) in private fp32 bins per lane and chunk
  // position, then reduce each in a fixed order in fp64, the wave that forms
  // a total posting it as word k of this workgroup's mailbox (buffer ppar,
  // step number pseq: the step that decides jn), and the sum of squares into
  // sh.wave_part if want_ssr.  The bins are cleared as they are read; an LDS
  // barrier separates the bin updates from the reduction.
  auto pass = [&](int ja, int jn, bool want_ssr, int lo, int ppar, uint32_t pseq) {
    const Ctx &ca = sh.ctx[(ja < 0 ? 0 : ja) & (kRing - 1)];
    const Ctx &cn = sh.ctx[(jn < 0 ? 0 : jn) & (kRing - 1)];
    const bool do_a = ja >= 0, do_n = jn >= 0;
    const int flags = sh.flags, acc = flags & 1, merged = (flags >> 1) & 1;
    const int kl = ca.pr.rank_l, kr = ca.pr.rank_r, eta_a = ca.pr.eta;
    const bool changed = do_a && acc && ca.pr.move != kNone;
    // a rejected GROW gives both children the merged value of eta (equal
    // deltas), so the predictor row that tells them apart is read only when
    // the GROW is accepted
    const bool xa = do_a && ca.pr.move == kGrow && acc, xn = do_n && cn.pr.move == kGrow;
    // the proposals' fields the per-chunk routes use, out of LDS once per pass
    // (read per chunk, each was a dependent LDS round trip, and its wait also
    // waited for the chunk's outstanding bin writes: n = 1e7, 215 -> 248
    // sweeps/s)
    const int eta_n = cn.pr.eta, cut_n = cn.pr.cut, grow_n = xn ? eta_n : -1;
    // a point of a GROW's eta goes right exactly when its rank is that of
    // the right child (every other slot has another rank), so the GROW
    // right-count is the number of bytes of the packed ranks equal to it;
    // without a GROW, a byte no rank takes (ranks: below kNullRank, or
    // kBadRank)
    static_assert(kNullRank < 254 && kBadRank != 254, "254 must be no rank");
    const uint32_t right4 = (uint32_t)(xn ? cn.rank_of[2 * eta_n + 1] : 254) * 0x01010101u;
    const int cut_a = ca.pr.cut, grow_a = do_a && ca.pr.move == kGrow ? eta_a : -1;
    const int n_obs = A->n;
    const uint32_t n_chunks = (uint32_t)A->chunks;
    // ranks of tree jn: computed from its rows by the first bin pass, read
    // back from the stash by the others
    const bool fresh = do_n && (!ST || lo == 0);
    const int Ln = do_n ? cn.pr.L : 0;
    // when tree jn's ranks all fit this pass but its last slot (lo == 0,
    // fewer leaves than the pass holds), every other rank (padding, an
    // inconsistent cache) goes to that spare slot, which no total reads and
    // the pass clears: no range test per point
    const bool spare = ST && lo == 0 && Ln < kPassRanks;
    // index rows of trees ja and jn: rows of the cache, or without one the
    // two rolling rows (by tree parity) that carry a tree's leaves from the
    // step that accumulates it to the step that applies it
    auto row_of = [&](int tree) {
      const int64_t r = CF ? (tree & 1) : tree;
      return gbl((ChunkT *)((char *)A->idx + r * A->ldi * IB));
    };
    const gptr<ChunkT> rowa = row_of(do_a ? ja : 0);
    const gptr<ChunkT> rown = row_of(do_n ? jn : 0);
    const bool trav = CF && do_n && lo == 0;  // Algorithm 1 for tree jn
    const NodeList &nn = sh.nl[(jn < 0 ? 0 : jn) & (kRing - 1)];
    // without an index cache: tree jn's internal-node count, its mask of
    // internal heap slots and its first 8 nodes (predictor-row offset, cut,
    // heap slot), out of LDS once per pass rather than per batch
    const int ni_p = trav ? nn.ni : 0;
    uint64_t imask_p = 0;
    int64_t xoff8[8];
    int cut8[8], slot8[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) xoff8[k] = 0, cut8[k] = 256, slot8[k] = 0;
    if (CF && trav && ni_p <= 32) {
      imask_p = nn.imask;
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (k < ni_p) {
          slot8[k] = nn.nh[k];
          cut8[k] = nn.cut8[k];
          xoff8[k] = (int64_t)nn.axis8[k] * A->ldx;
        }
    }
    // a tree's axis is read only when it takes part (a ring slot may not
    // hold a proposal yet); every proposal's axis is a valid row
    const gptr<const uint32_t> xra =
        gbl((const uint32_t *)(A->X + (int64_t)(do_a ? ca.pr.axis : 0) * A->ldx));
    const gptr<const uint32_t> xrn =
        gbl((const uint32_t *)(A->X + (int64_t)(do_n ? cn.pr.axis : 0) * A->ldx));
    const gptr<f32x4> res = gbl((f32x4 *)A->resid);
    double ssr = 0.0;
    int nr = 0;
    uint32_t bad = 0;
    // a batch of U chunks per thread: its loads, then its arithmetic; the
    // loop keeps the next two batches' loads in flight while one is computed
    struct Batch {
      uint32_t ch[U];        // chunk (unsigned: a 32-bit offset from a uniform base)
      int32_t sl[U];         // its stash word (-1: none)
      bool inl[U];           // the chunk's residuals are in LDS
      uint32_t ok[U];
      f32x4 rv[U];
      ChunkT ra[U], rn[U];
      uint32_t xa4[U], xn4[U];
    };
    // every lane issues every load, so each batch is the same fixed number
    // of loads and the compiler can wait for one batch while the next two
    // stay in flight (a skipped load would leave it unable to count them,
    // and it would drain them all); chunk 0 stands in for chunks past the
    // end and for a load whose value goes unused (one cached line per wave).
    // The arithmetic zeroes what a chunk past the end loaded, after which
    // its points are padding like those of a partial chunk (index entry 0,
    // residual 0)
    auto load_batch = [&](int i0, Batch &B) {
      uint32_t cu[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        B.ch[u] = (uint32_t)((w * cpt + i0 + u) * kBlock + t);
        B.sl[u] = i0 + u < cpt ? (i0 + u) * kBlock + t : -1;
        B.inl[u] = i0 + u < rc;
        const bool valid = i0 + u < cpt && B.ch[u] < n_chunks;
        const int32_t rem = n_obs - 4 * (int32_t)B.ch[u];
        B.ok[u] = !valid ? 0u : (rem >= 4 ? 15u : ((1u << rem) - 1u));
        cu[u] = valid ? B.ch[u] : 0u;
        B.rv[u] = res[B.inl[u] ? 0 : cu[u]];  // in LDS: chunk 0 stands in
      }
      // with the stash, tree ja's ranks come from LDS: no loads of its rows
      if (!ST) {
#pragma unroll
        for (int u = 0; u < U; ++u) B.ra[u] = rowa[do_a ? cu[u] : 0];
#pragma unroll
        for (int u = 0; u < U; ++u) B.xa4[u] = xra[xa ? cu[u] : 0];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) B.rn[u] = rown[fresh && !trav ? cu[u] : 0];
#pragma unroll
      for (int u = 0; u < U; ++u) B.xn4[u] = xrn[xn && fresh ? cu[u] : 0];
    };
    auto compute_batch = [&](Batch &B) {
      uint32_t (&ch)[U] = B.ch;
      uint32_t (&ok)[U] = B.ok;
      f32x4 (&rv)[U] = B.rv;
      ChunkT (&ra)[U] = B.ra;
      ChunkT (&rn)[U] = B.rn;
      uint32_t (&xa4)[U] = B.xa4;
      uint32_t (&xn4)[U] = B.xn4;
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (B.inl[u]) rv[u] = rcache[B.sl[u]];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (!ok[u]) {
          if (!ST) ra[u] = (ChunkT)0;
          rn[u] = (ChunkT)0;
          rv[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      if (trav && ni_p <= 32) {
        // leaves of tree jn by Algorithm 1 on its structure snapshot: the
        // decision of every internal node for the chunk's 4 points, from one
        // coalesced word of the node's predictor row (the words of up to 8
        // nodes in flight at a time, so a small tree costs one round trip,
        // not one per level), as a bit of a mask per point; then the descent
        // in registers (n = 1e7 without a cache: 68 sweeps/s level by level,
        // 90 with the masks, 99 with loads only for existing nodes and, up
        // to depth 6, bits by heap slot)
        uint32_t bits[U][4];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int b = 0; b < 4; ++b) bits[u][b] = 0u;
        const int ni = ni_p;
        const int H = A->H;
        // up to depth 6 the bit of a decision is its heap slot, and the
        // descent needs no LDS; deeper, it is the node's index in the list
        const bool by_slot = H <= 32;
        const uint64_t imask = imask_p;  // internal heap slots (by_slot)
        uint32_t cu[U];
#pragma unroll
        for (int u = 0; u < U; ++u) cu[u] = ok[u] ? ch[u] : 0u;
        for (int k0 = 0; k0 < ni; k0 += 8) {
          uint32_t wd[8][U];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
#pragma unroll
            for (int u = 0; u < U; ++u) wd[e][u] = 0u;
            if (k0 + e < ni) {
              const int64_t off = k0 == 0 ? xoff8[e] : (int64_t)cn.ax[nn.nh[k0 + e]] * A->ldx;
              const gptr<const uint32_t> xr = gbl((const uint32_t *)(A->X + off));
#pragma unroll
              for (int u = 0; u < U; ++u) wd[e][u] = xr[cu[u]];
            }
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int k = k0 + e;
            const int hk = k0 == 0 ? slot8[e] : (k < ni ? (int)nn.nh[k] : 0);
            // no bit past the last node
            const int cv = k0 == 0 ? cut8[e] : (k < ni ? (int)cn.ct[hk] : 256);
            const int pos = by_slot ? hk : (k & 31);
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
              for (int b = 0; b < 4; ++b)
                bits[u][b] |= (uint32_t)((int)((wd[e][u] >> (8 * b)) & 0xffu) >= cv) << pos;
          }
        }
        int hh[U][4];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int b = 0; b < 4; ++b) hh[u][b] = 1;
        if (by_slot) {
          for (int lvl = 1; lvl < A->D; ++lvl)
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
              for (int b = 0; b < 4; ++b) {
                const int h = hh[u][b];
                const bool in = (imask >> h) & 1ull;  // h < 64
                hh[u][b] = in ? 2 * h + (int)((bits[u][b] >> (h & 31)) & 1u) : h;
              }
        } else {
          for (int lvl = 1; lvl < A->D; ++lvl)
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
              for (int b = 0; b < 4; ++b) {
                const int h = hh[u][b];
                const int q = h < H ? (int)nn.nidx[h] : kNoNode;
                if (q != kNoNode) hh[u][b] = 2 * h + (int)((bits[u][b] >> q) & 1u);
              }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          ChunkT pk = 0;
#pragma unroll
          for (int b = 0; b < 4; ++b) pk = IC::put(pk, b, ((ok[u] >> b) & 1u) ? hh[u][b] : 0);
          rn[u] = pk;
          if (!ST && ok[u]) rown[ch[u]] = pk;
        }
      } else if (trav) {
        // a tree with more internal nodes than a mask holds (depth 8 only):
        // level by level, with the predictor bytes of all 4 U points in flight
        int hh[U][4];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int b = 0; b < 4; ++b) hh[u][b] = 1;
        const int H = A->H;
        for (int lvl = 1; lvl < A->D; ++lvl) {
          int xb[U][4];
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              const int h = hh[u][b];
              const int cv = h < H ? cn.ct[h] : 0;
              xb[u][b] = 0;
              if (((ok[u] >> b) & 1u) && cv)
                xb[u][b] = gbl(A->X)[(int64_t)cn.ax[h] * A->ldx + 4 * (int64_t)ch[u] + b];
            }
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              const int h = hh[u][b];
              const int cv = h < H ? cn.ct[h] : 0;
              if (cv) hh[u][b] = 2 * h + (xb[u][b] >= cv ? 1 : 0);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          ChunkT pk = 0;
#pragma unroll
          for (int b = 0; b < 4; ++b) pk = IC::put(pk, b, ((ok[u] >> b) & 1u) ? hh[u][b] : 0);
          rn[u] = pk;
          if (!ST && ok[u]) rown[ch[u]] = pk;
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (do_a) {
          uint32_t rk;
          if (ST)
            rk = ok[u] ? stash[B.sl[u]] : kNull4;
          else
            rk = ranks4(ca, grow_a, eta_a, cut_a, ra[u], xa4[u], bad, nullptr);
          float dl[4];
#pragma unroll
          for (int b = 0; b < 4; ++b) dl[b] = sh.dlt[(rk >> (8 * b)) & 0xff];
#pragma unroll
          for (int b = 0; b < 4; ++b) rv[u][b] += dl[b];  // final delta of the rank
          // the index row changes only under an accepted move
          bool touch = false;
          ChunkT out = 0;
          if (changed) {
            // every rank's heap slot read unconditionally (no exec mask per
            // point; ranks from kNullRank on have slot 0), then selected
            int hs[4];
#pragma unroll
            for (int b = 0; b < 4; ++b) hs[b] = ca.heap_of[(rk >> (8 * b)) & 0xff];
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              const int rnk = (rk >> (8 * b)) & 0xff;
              const bool pair = (rnk == kl) || (rnk == kr);
              touch |= pair;
              out = IC::put(out, b, (merged && pair) ? eta_a : hs[b]);
            }
          }
          if (B.inl[u])
            rcache[B.sl[u]] = rv[u];
          else if (ok[u])
            res[ch[u]] = rv[u];
          if (!CF && changed && touch && ok[u]) rowa[ch[u]] = out;
        }
        if (want_ssr) {
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const double x = (double)rv[u][b];  // 0 at padding points
            ssr += x * x;
          }
        }
        if (do_n) {
          // a private bin per lane and chunk position: the 4 points of a
          // chunk never share one, so the chunk is one batch of independent
          // read-modify-writes (chunks follow in LDS order); points of the
          // null rank or outside the pass go to the spare slot (spare) or add
          // 0 to a bin of the pass
          uint32_t rk;
          if (ST && lo > 0) {
            rk = ok[u] ? stash[B.sl[u]] : kNull4;
          } else {
            // (a uniform branch: a GROW's points of eta take a child; without
            // an index cache, the route of every pass measured faster)
            if (CF || !ST || xn)
              rk = ranks4(cn, grow_n, eta_n, cut_n, rn[u], xn4[u], bad, &nr);
            else
              rk = ranks4_plain(cn, rn[u], bad);
            if (ST && B.sl[u] >= 0) stash[B.sl[u]] = rk;  // after the read above
            if (ST) nr += zero_bytes(rk ^ right4);
          }
          // points b0..b0+kPos-1 go to kPos different bins, read together
          // and written together
          if (spare) {
#pragma unroll
            for (int b0 = 0; b0 < 4; b0 += kPos) {
              int q[kPos];
              float cur[kPos];
#pragma unroll
              for (int e = 0; e < kPos; ++e) {
                const uint32_t rl = min((rk >> (8 * (b0 + e))) & 0xffu, (uint32_t)(kPassRanks - 1));
                q[e] = ((((int)rl * kPos + e) * kWaves + wave) << 6) | lane;
              }
#pragma unroll
              for (int e = 0; e < kPos; ++e) cur[e] = sh.bins[q[e]];
#pragma unroll
              for (int e = 0; e < kPos; ++e) sh.bins[q[e]] = cur[e] + rv[u][b0 + e];
            }
          } else {
#pragma unroll
            for (int b0 = 0; b0 < 4; b0 += kPos) {
              int q[kPos];
              float add[kPos], cur[kPos];
#pragma unroll
              for (int e = 0; e < kPos; ++e) {
                const int rl = (int)((rk >> (8 * (b0 + e))) & 0xff) - lo;
                const bool in = rl >= 0 && rl < kPassRanks;
                q[e] = ((((in ? rl : 0) * kPos + e) * kWaves + wave) << 6) | lane;
                add[e] = in ? rv[u][b0 + e] : 0.f;
              }
#pragma unroll
              for (int e = 0; e < kPos; ++e) cur[e] = sh.bins[q[e]];
#pragma unroll
              for (int e = 0; e < kPos; ++e) sh.bins[q[e]] = cur[e] + add[e];
            }
          }
        }
      }
    };
    // batches past the last are loaded too (chunk 0, unused), so every
    // path through the loop issues the same loads
    Batch B0, B1, B2;
    load_batch(0, B0);
    load_batch(U, B1);
#pragma unroll 1
    for (int i0 = 0; i0 < cpt; i0 += 3 * U) {
      load_batch(i0 + 2 * U, B2);
      compute_batch(B0);
      if (i0 + U >= cpt) break;
      load_batch(i0 + 3 * U, B0);
      compute_batch(B1);
      if (i0 + 2 * U >= cpt) break;
      load_batch(i0 + 4 * U, B1);
      compute_batch(B2);
    }
    if (bad == kBadRank) sh.dev_err = 1;  // bad: the largest rank seen
    if (ST && do_n && lo == 0) {
      // per-lane counts (below 2^24) summed exactly over the wave
      const double tot = wave_total63((double)nr);
      if (lane == 63 && tot != 0.0) atomicAdd(&sh.nr[jn & 1], (int)tot);
    } else if (!ST && do_n && lo == 0 && lane == 0 && nr) {
      atomicAdd(&sh.nr[jn & 1], nr);  // wave-uniform
    }
    if (want_ssr) {
      const double tot = wave_total63(ssr);
      if (lane == 63) sh.wave_part[wave] = tot;
    }
    lds_barrier();
    if (do_n && lo == 0 && t == kBlock - 1) {
      // the GROW right-count of tree jn, complete after the barrier, as the
      // last word of this workgroup's mailbox for the step that decides jn
      post(A, sh, ppar, Ln, mk_word(pseq, (uint64_t)sh.nr[jn & 1]));
      sh.nr[jn & 1] = 0;
    }
    if (do_n) {
      if (spare && wave == (kPassRanks - 1) % kWaves)
#pragma unroll
        for (int u = 0; u < kWaves; ++u)
#pragma unroll
          for (int b = 0; b < kPos; ++b) sh.bins[((((kPassRanks - 1) * kPos + b) * kWaves + u) << 6) | lane] = 0.f;
      for (int k = lo + wave; k < min(Ln, lo + kPassRanks); k += kWaves) {
        double a = 0.0;
#pragma unroll
        for (int u = 0; u < kWaves; ++u)
#pragma unroll
          for (int b = 0; b < kPos; ++b) {
            const int q = ((((k - lo) * kPos + b) * kWaves + u) << 6) | lane;
            a += (double)sh.bins[q];
            sh.bins[q] = 0.f;
          }
        const double tot = wave_total63(a);
        // the wave that forms a total posts it
        if (lane == 63) post(A, sh, ppar, k, mk_word(pseq, pack_f64(tot)));
      }
    }
  };
  // all partial sums of tree jn: trees with more leaves than one bin pass
  // holds take extra accumulate-only passes over the data
  // (ppar, pseq: mailbox buffer and step number of the step that decides jn;
  // a pass that follows another waits for its bins to be cleared)
  auto pass_all = [&](int ja, int jn, bool want_ssr, int ppar, uint32_t pseq) {
    pass(ja, jn, want_ssr, 0, ppar, pseq);
    const int Ln = jn >= 0 ? sh.ctx[jn & (kRing - 1)].pr.L : 0;
    for (int lo = kPassRanks; lo < Ln; lo += kPassRanks) {
      lds_barrier();
      pass(-1, jn, false, lo, ppar, pseq);
    }
  };
  // axis and cut of one heap slot of tree j (thread t < H), packed
  auto struct_word = [&](int tree) -> uint32_t {
    const int H = A->H, h = t < H ? t : 0;
    const int64_t o = (int64_t)tree * H + h;
    return (uint32_t)gbl(A->axis)[o] | ((uint32_t)gbl(A->cut)[o] << 16);
  };
  auto store_struct = [&](Ctx &c, uint32_t wv) {
    if (t < A->H) {
      c.ax[t] = (uint16_t)(wv & 0xffffu);
      c.ct[t] = (uint8_t)(wv >> 16);
    }
  };
  // proposals of trees j0..j0+2, their rank tables (and structures, without
  // an index cache), the decision data of j0 and tree j0's partial sums
  auto refill = [&](int j0, int64_t s, int ppar, uint32_t pseq) {
    for (int q = 0; q < 3; ++q)
      if (j0 + q < m) {
        const uint32_t wd = load_prop_word(A, j0 + q);
        if (t < kPropWords) ((uint32_t *)&sh.ctx[(j0 + q) & (kRing - 1)].pr)[t] = wd;
        if (CF) store_struct(sh.ctx[(j0 + q) & (kRing - 1)], struct_word(j0 + q));
      }
    lds_barrier();
    for (int q = 0; q < 3; ++q)
      if (j0 + q < m) {
        build_ranks(A, sh.ctx[(j0 + q) & (kRing - 1)]);
        if (CF) build_inodes(A, sh.ctx[(j0 + q) & (kRing - 1)], sh.nl[(j0 + q) & (kRing - 1)]);
      }
    lds_barrier();
    const TdRegs tr0 = load_tree_data(A, sh.ctx[j0 & (kRing - 1)], j0, s);
    store_tree_data(sh.td[j0 & 1], sh.ctx[j0 & (kRing - 1)], tr0);
    pass_all(-1, j0, false, ppar, pseq);
  };

  // ---- prologue
  int64_t s = Lc.s0;
  int j = Lc.j0;
  if (j < m) {
    gen_proposals(A, seed, s, j);
    gen_normals(A, seed, s, j);
  }
  publish_workgroup();
  if (t == 0) post(A, sh, 1, 0, mk_word(1, 0));
  gather_total(A, sh, 1, 1, 0, Lc.spin_limit);
  // acquire by the wave that polled (a one-word gather polls on the last
  // wave); the barrier orders the other waves after it
  if (t >= kBlock - 64) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  __syncthreads();
  if (j < m && !sh.abort_flag) refill(j, s, 0, 2u);
  bool have_ssr = false;

#pragma unroll 1
  for (int step = 0; step < Lc.n_steps; ++step) {
    if (sh.abort_flag) break;
    const uint32_t seq = (uint32_t)step + 2;
    const int par = step & 1;
    if (j < m) {
      Ctx &c = sh.ctx[j & (kRing - 1)];
      const int L = c.pr.L;
      const bool more1 = (j + 1 < m) && (step + 1 < Lc.n_steps);
      const bool more3 = more1 && (j + 3 < m);
      const int j1 = more1 ? j + 1 : j, j3 = more3 ? j + 3 : j;
      const TdRegs tdn = load_tree_data(A, sh.ctx[j1 & (kRing - 1)], j1, s);
      const uint32_t pw3 = load_prop_word(A, j3);
      const uint32_t sw3 = CF ? struct_word(j3) : 0u;
      // with the stash, one word of every chunk of this step's first two
      // batches (residuals, index row and, for a GROW, predictor row of tree
      // j+1) is loaded now, while the grid exchanges the sums, so that those
      // batches come from the L2 when the pass starts after the decision
      // (n = 1e7: 194 -> 206 sweeps/s; one batch 203, three 197)
      constexpr int kTouch = (ST && !CF) ? 2 * U : 0;
      uint32_t touch[kTouch > 0 ? kTouch : 1][3];
      if (kTouch > 0) {
        const Ctx &cn = sh.ctx[j1 & (kRing - 1)];
        const bool xg = more1 && cn.pr.move == kGrow;
        const gptr<const uint32_t> rw = gbl((const uint32_t *)A->resid);
        const gptr<const uint32_t> nw =
            gbl((const uint32_t *)((const char *)A->idx + (int64_t)j1 * A->ldi * IB));
        const gptr<const uint32_t> xw =
            gbl((const uint32_t *)(A->X + (int64_t)cn.pr.axis * A->ldx));
#pragma unroll
        for (int u = 0; u < kTouch; ++u) {
          const int32_t ch = (w * cpt + u) * kBlock + t;
          const int32_t cu = (u < cpt && ch < A->chunks) ? ch : 0;
          touch[u][0] = rw[4 * (int64_t)(u < rc ? 0 : cu)];
          touch[u][1] = nw[IB * (int64_t)cu];
          touch[u][2] = xw[xg ? cu : 0];
        }
      }
      pre_decide(A, sh, c, sh.td[j & 1], w == 0 ? uncounted : -1);
      const int nseg = gather_polls(A, sh, par, seq, L + 1, L, Lc.spin_limit);
      // the touched words are discarded; issued before the polls, they have
      // arrived by the end of the gather, so this waits for nothing
#pragma unroll
      for (int u = 0; u < kTouch; ++u)
        asm volatile("" ::"v"(touch[u][0]), "v"(touch[u][1]), "v"(touch[u][2]));
      decide_step(A, sh, c, sh.td[j & 1], nseg);
      if (more3 && t < kPropWords) ((uint32_t *)&sh.ctx[(j + 3) & (kRing - 1)].pr)[t] = pw3;
      if (CF && more3) store_struct(sh.ctx[(j + 3) & (kRing - 1)], sw3);
      if (more1) store_tree_data(sh.td[(j + 1) & 1], sh.ctx[(j + 1) & (kRing - 1)], tdn);
      lds_barrier();
      finish_tree(A, Lc, sh, c, j, s, step);
      uncounted = j;
      if (more3) build_ranks(A, sh.ctx[(j + 3) & (kRing - 1)]);
      if (CF && more3) build_inodes(A, sh.ctx[(j + 3) & (kRing - 1)], sh.nl[(j + 3) & (kRing - 1)]);
      have_ssr = j == m - 1;
      pass_all(j, more1 ? j + 1 : -1, have_ssr, (step + 1) & 1, (uint32_t)step + 3);
      ++j;
    } else {
      if (w == 0 && t == kBlock - 1 && uncounted >= 0)
        count_move(sh, sh.ctx[uncounted & (kRing - 1)]);
      uncounted = -1;
      __syncthreads();
      if (!have_ssr) pass(-1, -1, true, 0, 0, 0u);
      have_ssr = false;
      sigma2_tail(A, Lc, sh, s, step, seq, par);
      if (A->probit) {
        const gptr<f32x4> res = gbl((f32x4 *)A->resid);
        for (int i0 = 0; i0 < cpt; ++i0) {
          const int32_t ch = (w * cpt + i0) * kBlock + t;
          if (ch >= A->chunks) break;
          const int32_t rem = A->n - 4 * ch;
          const uint32_t ok = rem >= 4 ? 15u : ((1u << rem) - 1u);
          const f32x4 rv = i0 < rc ? rcache[i0 * kBlock + t] : res[ch];
          float r4[4] = {rv[0], rv[1], rv[2], rv[3]};
          latent_chunk(A, seed, s, ch, ok, r4);
          if (i0 < rc)
            rcache[i0 * kBlock + t] = f32x4{r4[0], r4[1], r4[2], r4[3]};
          else
            res[ch] = f32x4{r4[0], r4[1], r4[2], r4[3]};
        }
      }
      j = 0;
      ++s;
      if (step + 1 < Lc.n_steps && !sh.abort_flag) refill(0, s, (step + 1) & 1, (uint32_t)step + 3);
    }
  }
  for (int i = 0; i < rc; ++i) {
    const int32_t ch = (w * cpt + i) * kBlock + t;
    if (ch < A->chunks) gbl((f32x4 *)A->resid)[ch] = rcache[i * kBlock + t];
  }
  if (w == 0 && t == kBlock - 1 && uncounted >= 0)
    count_move(sh, sh.ctx[uncounted & (kRing - 1)]);
  __syncthreads();
  if (w == 0 && t < 6) A->ctl->stats[t] += sh.stats[t];
  if (t == 0 && (sh.abort_flag || sh.dev_err))
    atomicOr(&A->ctl->error, (sh.abort_flag ? BART_DEVERR_TIMEOUT : 0u) |
                                 (sh.dev_err ? BART_DEVERR_CACHE : 0u));
}

template <int IB, bool CF, bool ST>
__global__ void __launch_bounds__(kBlock) sweep_kernel_stream(const SweepArgs *__restrict__ A,
                                                              Launch Lc) {
  __shared__ Shared sh;
  if ((int)blockIdx.x == Lc.absent_wg) return;
  const int c = (int)blockIdx.x / A->G;
  if (Lc.trace) Lc.trace += c * Lc.trace_stride;
  sweep_body_stream<IB, CF, ST>(A + c, Lc, sh);
}

}  // namespace bart
