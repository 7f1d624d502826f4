// featmap.h -- the Hedgehog feature map on a 32-row tile, cooperatively
// across the waves of a workgroup.
//
// phi(x) = [softmax(x W), softmax(-x W)] (Section 3.1), W in R^{d x F} per
// query head, f = 2F outputs.  For a tile X of 32 rows (queries or keys) the
// f outputs are cut into NPAIR = f/32 "pairs" (sign s, tile t): pair
// p = s*NT + t covers outputs s*F + 32t .. s*F + 32t + 31 and needs the
// product U^T tile t = W^T[32t .. 32t+31, :] X^T.  Pair p belongs to wave
// p % NW.  The softmax over the F entries of one sign spans NT pairs, so the
// row maxima and row sums go through LDS (two barriers).
//
// Operand convention: X arrives as the B operand of U^T = W^T X^T, i.e. lane
// (li, hh) holds row li of X and, for k-step ks, the entries
// ks*KW + hh*E + e.  The result register i of lane (li, hh) is feature
// row_of(i, hh) of the pair, for row li of X.
#pragma once

#include "device.h"

namespace hyb {

template <typename T, int D, int F, int NW>
struct FeatMap {
  typedef Mma<T> M;
  typedef typename M::op_t op_t;
  static constexpr int NT = F / kTile;     // U tiles
  static constexpr int NPAIR = 2 * NT;     // (sign, tile) pairs
  static constexpr int PPW = (NPAIR + NW - 1) / NW;
  static constexpr int KD = D / M::KW;     // k-steps over head_dim

  // LDS scratch: row maxima and row sums of each pair.
  struct alignas(16) Smem {
    float mx[NPAIR][kTile];
    float sm[NPAIR][kTile];
  };

  __device__ static inline bool owns(int w, int j) { return w + j * NW < NPAIR; }

  // A operands W_h^T[32t + li, :] of every pair this wave owns, loaded ahead
  // of use so that they are in flight together with the other block loads.
  __device__ static inline void load_w(const T* __restrict__ Wt_h, int w,
                                       int li, int hh,
                                       op_t (&wop)[PPW][KD]) {
#pragma unroll
    for (int j = 0; j < PPW; ++j) {
      if (!owns(w, j)) continue;
      const int t = (w + j * NW) % NT;
      const T* wrow = Wt_h + (size_t)(t * kTile + li) * D + hh * M::E;
#pragma unroll
      for (int ks = 0; ks < KD; ++ks) wop[j][ks] = load_op<T>(wrow + ks * M::KW);
    }
  }

  // U^T tile of every owned pair, negated for the second sign, and the
  // per-row maximum written to LDS.
  __device__ static inline void logits(const op_t (&wop)[PPW][KD],
                                       const op_t (&xop)[KD], int w, int li,
                                       int hh, float (&val)[PPW][16],
                                       Smem& sh) {
#pragma unroll
    for (int j = 0; j < PPW; ++j) {
      if (!owns(w, j)) continue;
      const int p = w + j * NW;
      const int sgn = p / NT;
      f32x16 acc = {};
#pragma unroll
      for (int ks = 0; ks < KD; ++ks) acc = M::mma(wop[j][ks], xop[ks], acc);
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        val[j][i] = sgn ? -acc[i] : acc[i];
        mx = fmaxf(mx, val[j][i]);
      }
      mx = fmaxf(mx, xor32(mx));
      if (hh == 0) sh.mx[p][li] = mx;
    }
  }

  // After a barrier: exponentials against the row maximum over all pairs
  // of the same sign, and per-pair row sums to LDS.
  __device__ static inline void exps(int w, int li, int hh,
                                     float (&val)[PPW][16], Smem& sh) {
#pragma unroll
    for (int j = 0; j < PPW; ++j) {
      if (!owns(w, j)) continue;
      const int p = w + j * NW;
      const int base = (p / NT) * NT;
      float mx = sh.mx[base][li];
#pragma unroll
      for (int t = 1; t < NT; ++t) mx = fmaxf(mx, sh.mx[base + t][li]);
      float s = 0.0f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        val[j][i] = fast_exp(val[j][i] - mx);
        s += val[j][i];
      }
      s += xor32(s);
      if (hh == 0) sh.sm[p][li] = s;
    }
  }

  // After a second barrier: normalise in place.  val[j][i] then holds
  // feature 32p + row_of(i, hh) of row li, p = w + j*NW (F = 32*NT, so the
  // pair index is also the 32-feature tile index).
  __device__ static inline void scale(int w, int li, float (&val)[PPW][16],
                                      const Smem& sh) {
#pragma unroll
    for (int j = 0; j < PPW; ++j) {
      if (!owns(w, j)) continue;
      const int p = w + j * NW;
      const int base = (p / NT) * NT;
      float s = 0.0f;
#pragma unroll
      for (int t = 0; t < NT; ++t) s += sh.sm[base + t][li];
      const float inv = 1.0f / s;
#pragma unroll
      for (int i = 0; i < 16; ++i) val[j][i] *= inv;
    }
  }

  // After a second barrier: normalise and hand every group of 4 consecutive
  // features of row li to store(first_feature, x[4]).
  template <typename Store>
  __device__ static inline void normalise(int w, int li, int hh,
                                          float (&val)[PPW][16], Smem& sh,
                                          Store store) {
#pragma unroll
    for (int j = 0; j < PPW; ++j) {
      if (!owns(w, j)) continue;
      const int p = w + j * NW;
      const int base = (p / NT) * NT;
      float s = 0.0f;
#pragma unroll
      for (int t = 0; t < NT; ++t) s += sh.sm[base + t][li];
      const float inv = 1.0f / s;
      const int f0 = (p / NT) * F + (p % NT) * kTile;
#pragma unroll
      for (int i = 0; i < 16; i += 4) {
        float x4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) x4[e] = val[j][i + e] * inv;
        store(f0 + row_of(i, hh), x4);  // 4 consecutive features
      }
    }
  }
};

// The whole feature map of one head inside one wave: no LDS, no barrier.
// The F/32 tiles of U^T = W_h^T X^T sit in this wave's accumulators, so both
// softmaxes (over the F entries of +U and of -U) reduce over registers and one
// cross-half exchange.  Output phi[p][i], p = s*NT + t: feature
// s*F + 32t + row_of(i, hh) of row li of X.
template <typename T, int D, int F>
struct WaveFeatMap {
  typedef Mma<T> M;
  typedef typename M::op_t op_t;
  static constexpr int NT = F / kTile;
  static constexpr int NPAIR = 2 * NT;
  static constexpr int KD = D / M::KW;

  // Feature index of flattened phi register j = 16p + i for lane half hh.
  __device__ __host__ static constexpr int feature(int j, int hh) {
    return (j / 16 / NT) * F + (j / 16 % NT) * kTile + row_of(j % 16, hh);
  }

  __device__ static inline void load_w(const T* __restrict__ Wt_h, int li,
                                       int hh, op_t (&wop)[NT][KD]) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const T* wrow = Wt_h + (size_t)(t * kTile + li) * D + hh * M::E;
#pragma unroll
      for (int ks = 0; ks < KD; ++ks) wop[t][ks] = load_op<T>(wrow + ks * M::KW);
    }
  }

  // The logits U^T = W^T X^T into phi[0 .. NT-1] (the operands of X are
  // free again afterwards).
  __device__ static inline void logits(const op_t (&wop)[NT][KD],
                                       const op_t (&xop)[KD],
                                       float (&phi)[NPAIR][16]) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      f32x16 acc = {};
#pragma unroll
      for (int ks = 0; ks < KD; ++ks) acc = M::mma(wop[t][ks], xop[ks], acc);
#pragma unroll
      for (int i = 0; i < 16; ++i) phi[t][i] = acc[i];
    }
  }

  // Both softmaxes over the logits.  keep = false gives phi = 0 (a padding
  // row) at no extra cost: it folds into the normalising factors.
  __device__ static inline void softmax(float (&phi)[NPAIR][16], bool keep) {
    float mx = -INFINITY, mn = INFINITY;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        mx = fmaxf(mx, phi[t][i]);
        mn = fminf(mn, phi[t][i]);
      }
    mx = fmaxf(mx, xor32(mx));
    mn = fminf(mn, xor32(mn));
    // e^(u - mx) = 2^(u log2 e - mx log2 e): one fma per exponent; the
    // rounding of mx log2 e is common to the row and cancels in the ratio
    constexpr float kLog2e = 1.4426950408889634f;
    const float mxl = mx * kLog2e, mnl = mn * kLog2e;
    float sp = 0.0f, sn = 0.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float u = phi[t][i];
        phi[t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(u, kLog2e, -mxl));       // softmax(+U)
        phi[NT + t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(-u, kLog2e, mnl));  // softmax(-U)
        sp += phi[t][i];
        sn += phi[NT + t][i];
      }
    sp += xor32(sp);
    sn += xor32(sn);
    const float ip = keep ? 1.0f / sp : 0.0f, in = keep ? 1.0f / sn : 0.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        phi[t][i] *= ip;
        phi[NT + t][i] *= in;
      }
  }

  __device__ static inline void compute(const op_t (&wop)[NT][KD],
                                        const op_t (&xop)[KD],
                                        float (&phi)[NPAIR][16],
                                        bool keep = true) {
    logits(wop, xop, phi);
    softmax(phi, keep);
  }
};

}  // namespace hyb
