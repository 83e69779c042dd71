// propose.hpp -- GROW/PRUNE proposal of one tree and the data-independent
// part of its Metropolis-Hastings log ratio, computed by one thread per tree.
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
#pragma once
#include "common.hpp"
#include "rng.hpp"

namespace bart {

__device__ __forceinline__ int depth_of(int h) { return 31 - __clz(h); }

__device__ __forceinline__ bool bit_get(const uint64_t (&m)[4], int h) {
  return (m[h >> 6] >> (h & 63)) & 1ull;
}
__device__ __forceinline__ void bit_set(uint64_t (&m)[4], int h) { m[h >> 6] |= 1ull << (h & 63); }
__device__ __forceinline__ void bit_clr(uint64_t (&m)[4], int h) {
  m[h >> 6] &= ~(1ull << (h & 63));
}
__device__ __forceinline__ int bits_below(const uint64_t (&m)[4], int h) {
  int r = 0;
  for (int k = 0; k < (h >> 6); ++k) r += __popcll(m[k]);
  if (h & 63) r += __popcll(m[h >> 6] & ((1ull << (h & 63)) - 1ull));
  return r;
}

// Bounds of node h on the (at most D-1 distinct) axes used by its ancestors.
struct Region {
  int n;
  int axis[8];
  int lo[8], hi[8];  // available cuts on axis[k] are lo+1..hi
};

__device__ inline void region_of(int h, const uint16_t *ax, const uint8_t *ct,
                                 const int32_t *n_cuts, Region &R) {
  R.n = 0;
  const int d = depth_of(h);
  for (int k = d; k >= 1; --k) {
    const int q = h >> k, child = h >> (k - 1);
    const int a = ax[q], s = ct[q];
    int e = -1;
    for (int u = 0; u < R.n; ++u)
      if (R.axis[u] == a) e = u;
    if (e < 0) {
      e = R.n++;
      R.axis[e] = a;
      R.lo[e] = 0;
      R.hi[e] = n_cuts[a];
    }
    if (child & 1)
      R.lo[e] = s;
    else
      R.hi[e] = s - 1;
  }
}

__device__ inline int exhausted(const Region &R) {
  int k = 0;
  for (int u = 0; u < R.n; ++u) k += (R.hi[u] - R.lo[u] <= 0);
  return k;
}

__device__ inline double psplit(const SweepArgs *__restrict__ A, int depth, int padj) {
  if (depth >= A->D - 1 || padj <= 0) return 0.0;
  return A->alpha * pow(1.0 + (double)depth, -A->beta);
}

__device__ inline double node_psplit(const SweepArgs *__restrict__ A, int h, const uint16_t *ax,
                                     const uint8_t *ct) {
  Region R;
  region_of(h, ax, ct, A->n_cuts, R);
  return psplit(A, depth_of(h), A->p_nz - exhausted(R));
}

__device__ inline double prob_grow(const SweepArgs *__restrict__ A, int nG, int nP) {
  return nP == 0 ? 1.0 : (nG == 0 ? 0.0 : A->p_grow);
}

// Proposal for tree j in sweep s from its current structure.
__device__ __noinline__ void propose_tree(const SweepArgs *__restrict__ A, Key key, int j,
                                          int64_t s, Prop &P) {
  const int H = A->H;
  const uint16_t *ax = A->axis + (int64_t)j * H;
  const uint8_t *ct = A->cut + (int64_t)j * H;

  // present nodes, leaves and prunable (nog) nodes, in increasing heap order
  uint64_t pres[4] = {0, 0, 0, 0}, leaf[4] = {0, 0, 0, 0};
  bit_set(pres, 1);
  int nG = 0, nP = 0;
  for (int h = 1; h < 2 * H; ++h) {
    if (!bit_get(pres, h)) continue;
    if (h < H && ct[h] != 0) {
      bit_set(pres, 2 * h);
      bit_set(pres, 2 * h + 1);
    } else {
      bit_set(leaf, h);
    }
  }
  for (int h = 1; h < 2 * H; ++h) {
    if (bit_get(leaf, h)) {
      nG += node_psplit(A, h, ax, ct) > 0.0;
    } else if (bit_get(pres, h) && bit_get(leaf, 2 * h) && bit_get(leaf, 2 * h + 1)) {
      ++nP;
    }
  }

  const Block b = draw(key, (uint64_t)s, (uint64_t)j, 0, 0);
  int move = kNone, eta = 0, a = 0, cut = 0;
  if (nG > 0 || nP > 0) {
    move = unit(b.w0) < prob_grow(A, nG, nP) ? kGrow : kPrune;
    if (move == kGrow) {
      int k = pick((uint32_t)b.w1, nG);
      for (int h = 1; h < 2 * H; ++h) {
        if (bit_get(leaf, h) && node_psplit(A, h, ax, ct) > 0.0) {
          if (k == 0) {
            eta = h;
            break;
          }
          --k;
        }
      }
      Region R;
      region_of(eta, ax, ct, A->n_cuts, R);
      // k-th available axis: the axes with cuts, minus those exhausted at eta
      int ex[8], nex = 0;
      for (int u = 0; u < R.n; ++u)
        if (R.hi[u] - R.lo[u] <= 0) ex[nex++] = A->nz_rank[R.axis[u]];
      for (int u = 1; u < nex; ++u)  // insertion sort by rank
        for (int v = u; v > 0 && ex[v - 1] > ex[v]; --v) {
          const int tmp = ex[v];
          ex[v] = ex[v - 1];
          ex[v - 1] = tmp;
        }
      int idx = pick((uint32_t)(b.w1 >> 32), A->p_nz - nex);
      for (int u = 0; u < nex; ++u) idx += (ex[u] <= idx);
      a = A->nz_list[idx];
      int lo = 0, hi = A->n_cuts[a];
      for (int u = 0; u < R.n; ++u)
        if (R.axis[u] == a) {
          lo = R.lo[u];
          hi = R.hi[u];
        }
      cut = lo + 1 + pick((uint32_t)b.w2, hi - lo);
    } else {
      int k = pick((uint32_t)b.w1, nP);
      for (int h = 1; h < H; ++h) {
        if (bit_get(pres, h) && !bit_get(leaf, h) && bit_get(leaf, 2 * h) &&
            bit_get(leaf, 2 * h + 1)) {
          if (k == 0) {
            eta = h;
            break;
          }
          --k;
        }
      }
    }
  }

  // count-free part of log r = log[pi(big)/pi(small)] + log[q(big->small)/q(small->big)];
  // the 1/(p_adj avail) factors of prior and proposal cancel
  double c_prior = 0.0;
  uint64_t big[4] = {leaf[0], leaf[1], leaf[2], leaf[3]};
  int rank_l = -1, rank_r = -1;
  if (move != kNone) {
    const int d = depth_of(eta);
    const bool sib_leaf = eta > 1 && bit_get(leaf, eta ^ 1);
    Region R;
    region_of(eta, ax, ct, A->n_cuts, R);
    const int padj_eta = A->p_nz - exhausted(R);
    const double ps_eta = psplit(A, d, padj_eta);
    double ps_l, ps_r;
    int nG_small, nP_small, nG_big, nP_big;
    if (move == kGrow) {
      int lo = 0, hi = A->n_cuts[a];
      for (int u = 0; u < R.n; ++u)
        if (R.axis[u] == a) {
          lo = R.lo[u];
          hi = R.hi[u];
        }
      ps_l = psplit(A, d + 1, padj_eta - ((cut - 1) - lo <= 0));
      ps_r = psplit(A, d + 1, padj_eta - (hi - cut <= 0));
      nG_small = nG;
      nP_small = nP;
      nG_big = nG - 1 + (ps_l > 0.0) + (ps_r > 0.0);
      nP_big = nP + 1 - (sib_leaf ? 1 : 0);
      bit_clr(big, eta);
      bit_set(big, 2 * eta);
      bit_set(big, 2 * eta + 1);
    } else {
      ps_l = node_psplit(A, 2 * eta, ax, ct);
      ps_r = node_psplit(A, 2 * eta + 1, ax, ct);
      nG_big = nG;
      nP_big = nP;
      nG_small = nG - (ps_l > 0.0) - (ps_r > 0.0) + (ps_eta > 0.0);
      nP_small = nP - 1 + (sib_leaf ? 1 : 0);
    }
    const double pg_small = prob_grow(A, nG_small, nP_small);
    const double pg_big = prob_grow(A, nG_big, nP_big);
    const double lr = log(ps_eta) - log(1.0 - ps_eta) + log(1.0 - ps_l) + log(1.0 - ps_r) +
                      log(1.0 - pg_big) - log((double)nP_big) - log(pg_small) +
                      log((double)nG_small);
    c_prior = move == kGrow ? lr : -lr;
    rank_l = bits_below(big, 2 * eta);
    rank_r = rank_l + 1;
  }
  int L = 0;
  for (int k = 0; k < 4; ++k) L += __popcll(big[k]);

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
  P.ln_u = log(unit(b.w3));
}

}  // namespace bart
