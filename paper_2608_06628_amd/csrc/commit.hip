// commit.hip -- fold a finished block into the recurrent state (Section 3.1
// state update): S_h += sum_t phi_h(k_t) v_t^T, z_h += sum_t phi_h(k_t).
//
// One workgroup per (request b, query head h); wave w of NW = D/32 owns the
// state columns 32w .. 32w+31 for all f rows.  The state tile is loaded
// straight into MFMA accumulator layout (row r = 32*rt + row_of(i, hh),
// column 32w + li), so S += phi(K)^T V is one accumulate-in-place product per
// 32-row tile, then stored back to the same addresses: every S element is read
// once and written once.  phi(K) is built with the shared feature-map code
// and transposed through LDS (feature-major) to serve as the A operand.
// On the bf16 path phi is kept as a bf16 pair hi + lo (two products), so the
// update carries phi to about 16 bits instead of 8.  Tokens beyond the
// request's block length get phi = 0 and v = 0 (padding rows are never used
// as values, whatever they hold).
#include "device.h"
#include "featmap.h"
#include "launch.h"

namespace hyb {

template <typename T, int D, int F>
struct CommitCfg {
  typedef Mma<T> M;
  typedef typename M::op_t op_t;
  static constexpr int NW = D / kTile;
  static constexpr int f = 2 * F;
  static constexpr int NRT = f / kTile;     // 32-row tiles of S
  static constexpr int KD = D / M::KW;
  static constexpr int KL = kTile / M::KW;  // k-steps over block tokens
  static constexpr int PT_LD = kTile + 16 / (int)sizeof(T);
  static constexpr int NPART = sizeof(T) == 2 ? 2 : 1;  // hi (+ lo) parts
  typedef FeatMap<T, D, F, NW> FM;
  struct alignas(16) Smem {
    T phiT[NPART][f][PT_LD];  // phi(k_t)[r] at [part][r][t]
    typename FM::Smem fm;
  };
};

template <typename T, int D, int F>
__global__ __launch_bounds__(kWave*(D / kTile)) void hyb_commit_kernel(
    CommitArgs a) {
  typedef CommitCfg<T, D, F> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  typedef typename C::FM FM;
  constexpr int f = C::f, E = M::E, KW = M::KW;
  __shared__ typename C::Smem sh;

  const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L;
  const int u = xcd_unit(blockIdx.x, a.s.B * Hq);
  const int b = u / Hq, h = u % Hq, g = h / (Hq / Hkv);
  const int slot = a.slots ? a.slots[b] : b;
  if (slot < 0 || slot >= a.s.n_slots) return;  // uniform per workgroup
  // Active tokens of this request's block (padding tokens contribute nothing).
  const int Lb = a.block_len ? min(max(a.block_len[b], 0), L) : L;
  if (Lb == 0) return;  // nothing to commit (uniform per workgroup)
  const size_t sbase = (size_t)slot * Hq + h;
  float* __restrict__ Sh = a.S + sbase * f * D;
  float* __restrict__ zh = a.z + sbase * f;
  const int col = w * kTile + li;

  // 1. Block operands, then z and the state tile (in accumulator layout),
  //    all unconditional and in bounds: padding tokens read row L-1 and are
  //    zeroed by a select.
  const size_t kstride = (size_t)Hkv * D;
  const T* __restrict__ Wt_h = (const T*)a.W + (size_t)h * F * D;
  op_t wop[FM::PPW][C::KD];
  FM::load_w(Wt_h, w, li, hh, wop);
  const T* __restrict__ kb = (const T*)a.k + ((size_t)b * L * Hkv + g) * D;
  const T* __restrict__ vb = (const T*)a.v + ((size_t)b * L * Hkv + g) * D;
  const bool tok_ok = li < Lb;
  op_t kop[C::KD];
  {
    const T* krow = kb + (size_t)min(li, Lb - 1) * kstride + hh * E;
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks) kop[ks] = load_op<T>(krow + ks * KW);
  }
  // V as B operand of phi^T V (k = token ks*KW + hh*E + e).
  op_t vop[C::KL];
#pragma unroll
  for (int ks = 0; ks < C::KL; ++ks)
    vop[ks] = load_rows_op<T>(vb + col, kstride, ks, hh, Lb, true);
  constexpr int NTH = kWave * C::NW, ZPT = (f + NTH - 1) / NTH;
  float zreg[ZPT];
#pragma unroll
  for (int j = 0; j < ZPT; ++j) zreg[j] = zh[min(tid + j * NTH, f - 1)];
  f32x16 sacc[C::NRT];
#pragma unroll
  for (int rt = 0; rt < C::NRT; ++rt)
#pragma unroll
    for (int j = 0; j < 4; ++j) {  // rows rt*32 + j*8 + hh*4 .. +3: 16 bytes
      const f32x4 x = *reinterpret_cast<const f32x4*>(
          Sh + (size_t)col * f + rt * kTile + row_of(4 * j, hh));
#pragma unroll
      for (int r = 0; r < 4; ++r) sacc[rt][4 * j + r] = x[r];
    }
#pragma unroll
  for (int ks = 0; ks < C::KD; ++ks) kop[ks] = keep_if<T>(tok_ok, kop[ks]);

  // 2. phi(K), transposed into LDS; padding tokens contribute nothing.
  float val[FM::PPW][16];
  FM::logits(wop, kop, w, li, hh, val, sh.fm);
  lds_barrier();
  FM::exps(w, li, hh, val, sh.fm);
  lds_barrier();
  FM::normalise(w, li, hh, val, sh.fm, [&](int f0, const float* x4) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x = tok_ok ? x4[e] : 0.0f;
      const T hi = from_f32<T>(x);
      sh.phiT[0][f0 + e][li] = hi;
      if constexpr (C::NPART == 2) sh.phiT[1][f0 + e][li] = from_f32<T>(x - to_f32(hi));
    }
  });
  lds_barrier();

  // 3. S += phi(K)^T V, one accumulate per 32-row tile, stored in place.
#pragma unroll
  for (int rt = 0; rt < C::NRT; ++rt) {
#pragma unroll
    for (int ks = 0; ks < C::KL; ++ks)
#pragma unroll
      for (int part = 0; part < C::NPART; ++part)
        sacc[rt] = M::mma(
            load_op<T>(&sh.phiT[part][rt * kTile + li][ks * KW + hh * E]),
            vop[ks], sacc[rt]);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<f32x4*>(Sh + (size_t)col * f + rt * kTile + row_of(4 * j, hh)) =
          f32x4{sacc[rt][4 * j], sacc[rt][4 * j + 1], sacc[rt][4 * j + 2], sacc[rt][4 * j + 3]};
  }

  // 4. z += sum_t phi(k_t), from the same values that entered S.
#pragma unroll
  for (int j = 0; j < ZPT; ++j) {
    const int r = tid + j * NTH;
    if (r >= f) continue;
    float s = 0.0f;
    for (int t = 0; t < Lb; ++t)
#pragma unroll
      for (int part = 0; part < C::NPART; ++part) s += to_f32(sh.phiT[part][r][t]);
    zh[r] = zreg[j] + s;
  }
}

template <typename T, int D, int F>
static hipError_t commit_go(const CommitArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((hyb_commit_kernel<T, D, F>), dim3(a.s.B * a.s.Hq),
                     dim3(kWave * (D / kTile)), 0, st, a);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t commit_f(const CommitArgs& a, hipStream_t st) {
  switch (a.s.F) {
    case 32: return commit_go<T, D, 32>(a, st);
    case 64: return commit_go<T, D, 64>(a, st);
    case 128: return commit_go<T, D, 128>(a, st);
  }
  return hipErrorInvalidValue;
}

template <typename T>
static hipError_t commit_d(const CommitArgs& a, hipStream_t st) {
  switch (a.s.D) {
    case 64: return commit_f<T, 64>(a, st);
    case 128: return commit_f<T, 128>(a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_commit(const CommitArgs& a, hipStream_t st) {
  return a.s.dtype == 1 ? commit_d<bf16>(a, st) : commit_d<float>(a, st);
}

}  // namespace hyb
