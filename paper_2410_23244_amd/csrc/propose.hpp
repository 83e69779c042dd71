// propose.hpp -- GROW/PRUNE proposal of one tree and the data-independent
// part of its Metropolis-Hastings log ratio, computed by one wave per tree.
//
// Sec. 3.3 ("Tree structure proposal", "Computations parallel across trees"):
// the move, the node and the splitting rule depend only on the tree and the
// random words, so all trees of a sweep are proposed together before the
// sequential tree loop, and the count-free terms of the acceptance ratio are
// computed there too.  The tree prior is the one of sec. 2.1: a node at
// depth d with an available split is internal with P_d = alpha (1+d)^-beta,
// its axis uniform over axes with an available split, its cut uniform over
// the available cuts; with the fixed maximum depth, nodes at depth D-1 are
// leaves (sec. 3.1, app. B).
//
// Wave layout: lane l holds internal heap slots l and l+64 (cut, the cut
// count of its axis, the axis, the rank of the axis among axes with cuts).
// Per-slot work (present, leaf, growable, prunable) runs one slot per lane
// with the ancestors fetched by lane permutes; the node choices are k-th
// set bits of wave ballots.  Everything is in registers: no scratch, and the
// only memory traffic is the tree's structure, its axes' cut counts and
// ranks, and the chosen axis.
#pragma once
#include "common.hpp"
#include "rng.hpp"

namespace bart {

constexpr int kMaxAnc = 7;  // ancestors of a node of a depth-8 tree

__device__ __forceinline__ int depth_of(int h) { return 31 - __clz(h); }

// bit h of a 256-bit mask held as four wave-uniform words; h may vary by lane
__device__ __forceinline__ int bit4(const uint64_t (&m)[4], int h) {
  const int k = h >> 6;
  const uint64_t w = k == 0 ? m[0] : k == 1 ? m[1] : k == 2 ? m[2] : m[3];
  return (int)((w >> (h & 63)) & 1ull);
}

// number of set bits of m below bit h
__device__ __forceinline__ int bits_below(const uint64_t (&m)[4], int h) {
  int r = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int sh = h - 64 * k;  // bits of word k below h: min(max(sh, 0), 64)
    const uint64_t part = sh >= 64 ? m[k] : (sh <= 0 ? 0ull : m[k] & ((1ull << sh) - 1ull));
    r += __popcll(part);
  }
  return r;
}

// Internal-node words of one tree: cut (bits 0-7), cut count of the node's
// axis (8-15), axis (16-31); slot l in w0, slot l+64 in w1 of lane l.
struct TreeRegs {
  uint32_t w0, w1;
  int32_t r0, r1;  // rank of the node's axis among the axes with cuts
};

__device__ __forceinline__ int wd_cut(uint32_t w) { return (int)(w & 0xffu); }
__device__ __forceinline__ int wd_nc(uint32_t w) { return (int)((w >> 8) & 0xffu); }
__device__ __forceinline__ int wd_axis(uint32_t w) { return (int)(w >> 16); }

// word of internal slot q (1 <= q < H, lane-varying allowed)
__device__ __forceinline__ uint32_t node_word(const TreeRegs &T, int q, int H) {
  const uint32_t a = (uint32_t)__shfl((int)T.w0, q & 63);
  if (H <= 64) return a;
  const uint32_t b = (uint32_t)__shfl((int)T.w1, q & 63);
  return q < 64 ? a : b;
}
__device__ __forceinline__ int node_rank(const TreeRegs &T, int q, int H) {
  const int a = __shfl(T.r0, q & 63);
  if (H <= 64) return a;
  const int b = __shfl(T.r1, q & 63);
  return q < 64 ? a : b;
}

// The path to node h: ancestor i (i = 0 the parent) is heap slot h >> (i+1),
// and h descends to its right child iff bit i of h is set.
struct Anc {
  uint32_t w[kMaxAnc];
  int d;  // depth of h = number of ancestors
};

__device__ __forceinline__ Anc ancestors(const TreeRegs &T, int h, int H) {
  Anc P;
  P.d = depth_of(h);
#pragma unroll
  for (int i = 0; i < kMaxAnc; ++i) P.w[i] = node_word(T, i < P.d ? h >> (i + 1) : 1, H);
  return P;
}

__device__ __forceinline__ bool path_present(const Anc &P) {
  bool ok = true;
#pragma unroll
  for (int i = 0; i < kMaxAnc; ++i) ok = ok && (i >= P.d || wd_cut(P.w[i]) != 0);
  return ok;
}

// Cuts of axis a still available below the path: lo+1..hi, starting from
// 0..n_a and narrowing from the root down (a right turn at cut c sets
// lo = c, a left turn sets hi = c - 1).
__device__ __forceinline__ void path_bounds(const Anc &P, int h, int a, int &lo, int &hi) {
#pragma unroll
  for (int i = kMaxAnc - 1; i >= 0; --i) {
    if (i < P.d && wd_axis(P.w[i]) == a) {
      if ((h >> i) & 1)
        lo = wd_cut(P.w[i]);
      else
        hi = wd_cut(P.w[i]) - 1;
    }
  }
}

// Which ancestors carry the root-most use of an axis whose available cuts
// are exhausted at h (bit i set for ancestor i); the number of such axes is
// the count of axes with no split left at h.
__device__ __forceinline__ uint32_t exhausted_set(const Anc &P, int h) {
  uint32_t e = 0;
#pragma unroll
  for (int u = 0; u < kMaxAnc; ++u) {
    const int a = wd_axis(P.w[u]);
    bool rep = u < P.d;
#pragma unroll
    for (int v = u + 1; v < kMaxAnc; ++v) rep = rep && !(v < P.d && wd_axis(P.w[v]) == a);
    int lo = 0, hi = wd_nc(P.w[u]);
    path_bounds(P, h, a, lo, hi);
    e |= (rep && hi - lo <= 0 ? 1u : 0u) << u;
  }
  return e;
}

// exhausted_set for a wave-uniform path (the node of the move): lane u < 7
// takes ancestor u; all 64 lanes must call it
__device__ __forceinline__ uint32_t exhausted_set_wave(const Anc &P, int h) {
  const int u = threadIdx.x & 63;
  uint32_t wu = P.w[0];
#pragma unroll
  for (int i = 1; i < kMaxAnc; ++i) wu = u == i ? P.w[i] : wu;
  const int a = wd_axis(wu);
  bool rep = u < P.d;
  int lo = 0, hi = wd_nc(wu);
#pragma unroll
  for (int v = kMaxAnc - 1; v >= 0; --v) {
    const bool same = v < P.d && wd_axis(P.w[v]) == a;
    rep = rep && !(v > u && same);
    if (same) {
      if ((h >> v) & 1)
        lo = wd_cut(P.w[v]);
      else
        hi = wd_cut(P.w[v]) - 1;
    }
  }
  return (uint32_t)__ballot(rep && hi - lo <= 0) & ((1u << kMaxAnc) - 1u);
}

__device__ __forceinline__ double prob_grow(const SweepArgs *__restrict__ A, int nG, int nP) {
  return nP == 0 ? 1.0 : (nG == 0 ? 0.0 : A->p_grow);
}

// alpha (1+d)^-beta for d = 0..7, wave-uniform
struct SplitTab {
  double v[8];
};

// P_d, or 0 at the depth limit or without an available axis (depth may vary
// by lane; no cross-lane operation, so it is safe under divergence)
__device__ __forceinline__ double psplit(const SweepArgs *__restrict__ A, const SplitTab &tb,
                                         int depth, int padj) {
  double v = tb.v[0];
#pragma unroll
  for (int d = 1; d < 8; ++d) v = depth == d ? tb.v[d] : v;
  return depth >= A->D - 1 || padj <= 0 ? 0.0 : v;
}

// Heap slot of the k-th (from 0) set bit of m over the first nw words;
// k is wave-uniform and smaller than the number of set bits.
__device__ __forceinline__ int kth_bit(const uint64_t (&m)[4], int nw, int k) {
  const int l = threadIdx.x & 63;
  uint64_t w = 0;
  int base = 0;
  bool found = false;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int c = __popcll(m[r]);
    if (!found && r < nw) {
      if (k < c || r == nw - 1) {
        w = m[r];
        base = 64 * r;
        found = true;
      } else {
        k -= c;
      }
    }
  }
  const uint64_t below = l ? w & ((1ull << l) - 1ull) : 0ull;
  const uint64_t b = __ballot(((w >> l) & 1ull) && __popcll(below) == k);
  return base + __ffsll((long long)b) - 1;
}

// Proposal for tree j in sweep s from its current structure; called by all
// 64 lanes of a wave with the same j, lane 0 writes P.
__device__ __noinline__ void propose_tree(const SweepArgs *__restrict__ A, Key key, int j,
                                          int64_t s, Prop &P) {
  const int H = A->H, l = threadIdx.x & 63;
  const gptr<const uint16_t> ax = gbl((const uint16_t *)A->axis) + (int64_t)j * H;
  const gptr<const uint8_t> ct = gbl((const uint8_t *)A->cut) + (int64_t)j * H;
  const gptr<const int32_t> ncut = gbl(A->n_cuts);
  const gptr<const int32_t> nzr = gbl(A->nz_rank);

  TreeRegs T;
  {
    const int c0 = l < H ? ct[l] : 0, c1 = l + 64 < H ? ct[l + 64] : 0;
    const int a0 = l < H ? ax[l] : 0, a1 = l + 64 < H ? ax[l + 64] : 0;
    const bool v0 = c0 != 0 && a0 < A->p, v1 = c1 != 0 && a1 < A->p;
    const int n0 = v0 ? ncut[a0] : 0, n1 = v1 ? ncut[a1] : 0;
    T.r0 = v0 ? nzr[a0] : -1;
    T.r1 = v1 ? nzr[a1] : -1;
    T.w0 = (uint32_t)c0 | (uint32_t)n0 << 8 | (uint32_t)a0 << 16;
    T.w1 = (uint32_t)c1 | (uint32_t)n1 << 8 | (uint32_t)a1 << 16;
  }
  SplitTab tab;
  {
    const double own = l < 8 ? A->alpha * pow(1.0 + (double)l, -A->beta) : 0.0;
#pragma unroll
    for (int d = 0; d < 8; ++d) tab.v[d] = __shfl(own, d);
  }

  // at most d distinct axes are used above a node of depth d, so with
  // p_nz >= D-1 every node above the depth limit keeps an available axis
  const bool all_avail = A->p_nz >= A->D - 1;

  // present nodes, leaves and growable leaves, one heap slot per lane
  const int nw = (2 * H + 63) >> 6;
  uint64_t pres[4] = {0, 0, 0, 0}, leaf[4] = {0, 0, 0, 0}, grow[4] = {0, 0, 0, 0};
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (r >= nw) break;
    const int h = 64 * r + l;
    const bool slot = h >= 1 && h < 2 * H;
    const int hh = slot ? h : 1;
    const Anc Pa = ancestors(T, hh, H);
    const bool present = slot && path_present(Pa);
    const uint32_t own = r == 0 ? T.w0 : (r == 1 ? T.w1 : 0u);
    const bool is_leaf = present && (h >= H || wd_cut(own) == 0);
    const int padj = all_avail ? A->p_nz : A->p_nz - __popc(exhausted_set(Pa, hh));
    const bool g = is_leaf && psplit(A, tab, Pa.d, padj) > 0.0;
    pres[r] = __ballot(present);
    leaf[r] = __ballot(is_leaf);
    grow[r] = __ballot(g);
  }
  // prunable nodes: present internal nodes whose two children are leaves
  uint64_t nog[4] = {0, 0, 0, 0};
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (r >= nw) break;
    const int h = 64 * r + l;
    const bool c = h >= 1 && h < H && bit4(pres, h) && !bit4(leaf, h) && bit4(leaf, 2 * h) &&
                   bit4(leaf, 2 * h + 1);
    nog[r] = __ballot(c);
  }
  int nG = 0, nP = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    nG += __popcll(grow[r]);
    nP += __popcll(nog[r]);
  }

  const Block b = draw(key, (uint64_t)s, (uint64_t)j, 0, 0);
  int move = kNone, eta = 0, a = 0, cut = 0;
  double c_prior = 0.0;
  uint64_t big[4] = {leaf[0], leaf[1], leaf[2], leaf[3]};
  int rank_l = -1, rank_r = -1;
  // arguments of the logarithms of the count-free ratio (1 when unused)
  double ps_eta = 1.0, ps_l = 0.0, ps_r = 0.0, pg_small = 1.0, pg_big = 0.0;
  int nG_small = 1, nP_big = 1;
  if (nG > 0 || nP > 0) {
    move = unit(b.w0) < prob_grow(A, nG, nP) ? kGrow : kPrune;
    uint64_t cand[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) cand[r] = move == kGrow ? grow[r] : nog[r];
    eta = kth_bit(cand, nw, pick((uint32_t)b.w1, move == kGrow ? nG : nP));
    const Anc Pe = ancestors(T, eta, H);
    const int d = Pe.d;
    // a PRUNE needs only the sign of P_d at eta, known when every node keeps an axis
    const uint32_t ex = move == kGrow || !all_avail ? exhausted_set_wave(Pe, eta) : 0u;
    const int nex = __popc(ex);
    const int padj_eta = A->p_nz - nex;
    ps_eta = psplit(A, tab, d, padj_eta);
    const bool sib_leaf = eta > 1 && bit4(leaf, eta ^ 1);
    int nP_small, nG_big;
    if (move == kGrow) {
      // the idx0-th axis with cuts that is not exhausted at eta: skipping the
      // exhausted ranks in increasing order (each at or below the running
      // index moves it up by one) ends at the least r >= idx0 with
      // r = idx0 + #{exhausted ranks <= r}, which lies in idx0..idx0+7;
      // lane c tests r = idx0 + c
      const int idx0 = pick((uint32_t)(b.w1 >> 32), padj_eta);
      int rk[kMaxAnc];
#pragma unroll
      for (int u = 0; u < kMaxAnc; ++u) rk[u] = node_rank(T, u < d ? eta >> (u + 1) : 1, H);
      const int rc = idx0 + l;
      int below = 0;
#pragma unroll
      for (int u = 0; u < kMaxAnc; ++u) below += (((ex >> u) & 1u) && rk[u] <= rc) ? 1 : 0;
      const uint64_t fixed = __ballot(l <= kMaxAnc && idx0 + below == rc);
      const int idx = idx0 + __ffsll((long long)fixed) - 1;
      a = gbl(A->nz_list)[idx];
      int lo = 0, hi = ncut[a];
      path_bounds(Pe, eta, a, lo, hi);
      cut = lo + 1 + pick((uint32_t)b.w2, hi - lo);
      ps_l = psplit(A, tab, d + 1, padj_eta - ((cut - 1) - lo <= 0));
      ps_r = psplit(A, tab, d + 1, padj_eta - (hi - cut <= 0));
      nG_small = nG;
      nP_small = nP;
      nG_big = nG - 1 + (ps_l > 0.0) + (ps_r > 0.0);
      nP_big = nP + 1 - (sib_leaf ? 1 : 0);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (r == eta >> 6) big[r] &= ~(1ull << (eta & 63));
        if (r == (2 * eta) >> 6) big[r] |= 3ull << ((2 * eta) & 63);
      }
    } else {
      const Anc Pl = ancestors(T, 2 * eta, H), Pr = ancestors(T, 2 * eta + 1, H);
      ps_l = psplit(A, tab, d + 1,
                    all_avail ? A->p_nz : A->p_nz - __popc(exhausted_set_wave(Pl, 2 * eta)));
      ps_r = psplit(A, tab, d + 1,
                    all_avail ? A->p_nz : A->p_nz - __popc(exhausted_set_wave(Pr, 2 * eta + 1)));
      nG_big = nG;
      nP_big = nP;
      nG_small = nG - (ps_l > 0.0) - (ps_r > 0.0) + (ps_eta > 0.0);
      nP_small = nP - 1 + (sib_leaf ? 1 : 0);
    }
    pg_small = prob_grow(A, nG_small, nP_small);
    pg_big = prob_grow(A, nG_big, nP_big);
    rank_l = bits_below(big, 2 * eta);
    rank_r = rank_l + 1;
  }
  // count-free part of log r = log[pi(big)/pi(small)] + log[q(big->small)/q(small->big)]
  // (the 1/(p_adj avail) factors of prior and proposal cancel), its eight
  // logarithms one per lane and summed in a fixed order; lane 8 the log of
  // the accept uniform
  double arg = unit(b.w3);
  arg = l == 0 ? ps_eta : arg;
  arg = l == 1 ? 1.0 - ps_eta : arg;
  arg = l == 2 ? 1.0 - ps_l : arg;
  arg = l == 3 ? 1.0 - ps_r : arg;
  arg = l == 4 ? 1.0 - pg_big : arg;
  arg = l == 5 ? (double)nP_big : arg;
  arg = l == 6 ? pg_small : arg;
  arg = l == 7 ? (double)nG_small : arg;
  const double lg = log(arg);
  const double lr = __shfl(lg, 0) - __shfl(lg, 1) + __shfl(lg, 2) + __shfl(lg, 3) +
                    __shfl(lg, 4) - __shfl(lg, 5) - __shfl(lg, 6) + __shfl(lg, 7);
  const double ln_u = __shfl(lg, 8);
  if (move != kNone) c_prior = move == kGrow ? lr : -lr;
  int L = 0;
  for (int k = 0; k < 4; ++k) L += __popcll(big[k]);

  if (l == 0) {
    P.move = move;
    P.eta = eta;
    P.axis = a;
    P.cut = cut;
    P.nG = nG;
    P.nP = nP;
    P.L = L;
    P.rank_l = rank_l;
    P.rank_r = rank_r;
    P.pad0 = P.pad1 = P.pad2 = 0;
    for (int k = 0; k < 4; ++k) P.mask[k] = big[k];
    P.c_prior = c_prior;
    P.ln_u = ln_u;
  }
}

}  // namespace bart
