// rng.hpp -- counter-based random numbers for the BART sweep on gfx950.
//
// The paper pre-generates every random number of a sweep as standard
// uniforms and normals and transforms them later (sec. 3.3, "Computations
// parallel across trees", item 5).  Here each draw is a pure function of
// (seed, chain, sweep s, tree j, purpose q, slot t) through Philox4x64-10
// (Salmon, Moraes, Dror and Shaw, SC'11): any workgroup can regenerate any
// draw, so redundant per-workgroup decisions agree bit for bit.
//
// Stream layout (counter words c0..c3, key (seed, 0x42415254)) of chain c,
// with C = c 2^32 (every t below is < 2^32, so chains never share a
// counter, and chain 0 of a batch draws exactly what a lone chain draws):
//   (s, j, 0, C)       proposal words of tree j in sweep s:
//                        w0 -> u_move, lo32(w1) -> node pick,
//                        hi32(w1) -> axis pick, lo32(w2) -> cut pick,
//                        w3 -> u_accept
//   (s, j, 1, C + u)   the leaf normals of heap slots 2u (w0,w1), 2u+1 (w2,w3)
//   (s, ~0, 2, C + t)  attempt t of the sigma^2 gamma draw
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bart {

struct Block {
  uint64_t w0, w1, w2, w3;
};

constexpr uint64_t kKeyTag = 0x42415254ull;

// Random stream of one chain: the seed and the chain's offset of the last
// counter word.
struct Key {
  uint64_t seed, chain_hi;
};

__device__ __forceinline__ Key chain_key(uint64_t seed, int chain) {
  return Key{seed, (uint64_t)(uint32_t)chain << 32};
}

__device__ __forceinline__ Block philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2,
                                               uint64_t c3, uint64_t k0, uint64_t k1) {
  // round function: two 64x64 -> 128 products, Weyl-sequence key schedule
  constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += W0;
      k1 += W1;
    }
    const uint64_t lo0 = M0 * c0, hi0 = __umul64hi(M0, c0);
    const uint64_t lo1 = M1 * c2, hi1 = __umul64hi(M1, c2);
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return Block{c0, c1, c2, c3};
}

__device__ __forceinline__ Block draw(Key key, uint64_t s, uint64_t j, uint64_t q, uint64_t t) {
  return philox4x64_10(s, j, q, key.chain_hi + t, key.seed, kKeyTag);
}

// (k + 1/2) 2^-52 with k the top 52 bits: exact in fp64, strictly in (0,1)
__device__ __forceinline__ double unit(uint64_t w) {
  return ((double)(w >> 12) + 0.5) * 0x1.0p-52;
}

// index in [0, k) by 32x32 -> 64 multiply-shift (no rejection step)
__device__ __forceinline__ int pick(uint32_t w, int k) {
  return (int)(((uint64_t)w * (uint64_t)(uint32_t)k) >> 32);
}

// Box-Muller, cosine branch
__device__ __forceinline__ double gauss(uint64_t a, uint64_t b) {
  const double two_pi = 6.283185307179586;  // fp64 nearest to 2 pi
  return sqrt(-2.0 * log(unit(a))) * cos(two_pi * unit(b));
}

// Gamma(shape, 1), shape >= 1, by Marsaglia and Tsang (2000): squeeze-free
// acceptance test on log u.  Bounded number of attempts.
__device__ __noinline__ double gamma_mt(Key key, uint64_t s, double shape) {
  const double d = shape - 1.0 / 3.0;
  const double c = 1.0 / sqrt(9.0 * d);
  for (uint64_t t = 0; t < 4096; ++t) {
    const Block b = draw(key, s, ~0ull, 2, t);
    const double z = gauss(b.w0, b.w1);
    const double u = unit(b.w2);
    double v = 1.0 + c * z;
    v = v * v * v;
    if (v > 0.0 && log(u) < 0.5 * z * z + d - d * v + d * log(v)) return d * v;
  }
  return d;
}

}  // namespace bart
