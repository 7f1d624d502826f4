// commit.hip -- fold a finished block into the recurrent state (Section 3.1
// state update): S_h += sum_t phi_h(k_t) v_t^T, z_h += sum_t phi_h(k_t).
//
// One workgroup per (request b, query head h); wave w of NW = D/32 owns the
// state columns 32w .. 32w+31 for all f rows, i.e. 32 consecutive rows of
// the stored S_h^T ([d][f], features contiguous): a contiguous 16 KiB.  The
// update is formed transposed, S^T += V^T phi(K), so the accumulator tile
// (w, rt) holds value dim c = 32w + row_of(i, hh) in register i and feature
// r = 32 rt + li in lane li: the state moves in and out with 4-byte accesses
// whose 32 lanes cover a whole 128-byte line, two lines per instruction.
// (With features in registers instead, every 16-byte access of an
// instruction would land in a different line; that costs a fifth of the
// bandwidth of a read-modify-write stream on this chip.)  Every S element is
// read once and written once.  phi(K) is built with the shared feature-map
// code and stored feature-major in LDS, the B operand of the update.
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
__global__ __launch_bounds__(kWave*(D / kTile), 2) void hyb_commit_kernel(
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
  // (slot and block length are uniform: through readfirstlane the state's
  // base address is a scalar, and each state access needs only a 32-bit
  // lane offset and an immediate, not a 64-bit address of its own)
  const int slot = __builtin_amdgcn_readfirstlane(a.slots ? a.slots[b] : b);
  if (slot < 0 || slot >= a.s.n_slots) return;  // uniform per workgroup
  // Active tokens of this request's block (padding tokens contribute nothing).
  const int Lb = __builtin_amdgcn_readfirstlane(a.block_len ? min(max(a.block_len[b], 0), L) : L);
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
#pragma unroll
  for (int ks = 0; ks < C::KD; ++ks) kop[ks] = keep_if<T>(tok_ok, kop[ks]);

  // 2. phi(K), transposed into LDS; padding tokens contribute nothing.  The
  //    state is requested after the logits, when the W_h and K operands are
  //    no longer live (their loads are not queued behind the state reads).
  float val[FM::PPW][16];
  FM::logits(wop, kop, w, li, hh, val, sh.fm);
  asm volatile("" ::: "memory");  // the state loads stay after the logits
  // tile (w, rt): value dim 32w + row_of(i, hh), feature 32 rt + li
  f32x16 sacc[C::NRT];
  // Buffer accesses over this head's state: the lane offset in one VGPR,
  // the 8-row group of register i in the scalar offset, the rest in the
  // immediate.
  const __amdgpu_buffer_rsrc_t srs =
      __builtin_amdgcn_make_buffer_rsrc(Sh, 0, f * D * 4, kBufferWord3);
  const int soff = ((w * kTile + hh * 4) * f + li) * 4;  // bytes
#pragma unroll
  for (int rt = 0; rt < C::NRT; ++rt)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      sacc[rt][i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
          srs, soff + ((i & 3) * f + rt * kTile) * 4, (i >> 2) * 8 * f * 4, 0));
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

  // 3. S^T += V^T phi(K), one accumulate per 32-feature tile, stored in place.

#pragma unroll
  for (int rt = 0; rt < C::NRT; ++rt) {
#pragma unroll
    for (int ks = 0; ks < C::KL; ++ks)
#pragma unroll
      for (int part = 0; part < C::NPART; ++part)
        sacc[rt] = M::mma(vop[ks],
                          load_op<T>(&sh.phiT[part][rt * kTile + li][ks * KW + hh * E]),
                          sacc[rt]);
#pragma unroll
    for (int i = 0; i < 16; ++i)
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, (float)sacc[rt][i]), srs,
                                            soff + ((i & 3) * f + rt * kTile) * 4,
                                            (i >> 2) * 8 * f * 4, 0);
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
  if (commit_grouped_supported(a.s)) return launch_commit_grouped(a, st);
  return a.s.dtype == 1 ? commit_d<bf16>(a, st) : commit_d<float>(a, st);
}

}  // namespace hyb
