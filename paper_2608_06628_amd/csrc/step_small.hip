// step_small.hip -- the hybrid step (Section 3.1: within-block softmax,
// linear readout of the committed state, gated merge with a shared
// normaliser) for batches too small to fill the chip with one workgroup per
// group of query heads.
//
// One wave per (request b, query head h, 32-column slice s of the head
// dimension).  Each wave forms everything its columns need -- the block
// scores and their softmax over the L keys, phi(Q) and lin_den = phi(Q) z,
// the merge coefficients -- and then only its slice of the two products:
// a P V[:, slice] and b phi(Q) S[:, slice].  The per-query work (scores,
// feature map, coefficients) is repeated by the D/32 slices of a head; in
// exchange a head's 64 KiB state is read by D/32 waves at once, which is what
// a batch of a few requests needs to reach the memory system from many CUs.
// At B = 8 (16 query heads, d = 128) that is 512 waves instead of 32
// workgroups.
//
// Layout of every product: 32x32 MFMA tiles, results transposed (rows =
// the slice's columns, columns = queries), so each lane owns one query and
// the merge coefficients are per-lane scalars.  The scores are formed as
// K Q^T (keys in rows), the softmax reduces over registers and one
// cross-half exchange, and the P V product takes P straight from the score
// accumulators (keys in accumulator-row order, the same order in which the
// V^T operand gathers its keys).  phi(Q) comes from the one-wave feature map
// (featmap.h), whose registers are read as the readout's B operand, features
// in accumulator-row order; the state operand reads the same features: two
// runs of four consecutive fp32 values per lane and k-step, rounded to the
// operand type.  As in the main step kernel, phi(Q) and the state enter the
// readout as bf16 on the bf16 path, and P as a bf16 pair hi + lo.
#include "device.h"
#include "featmap.h"
#include "launch.h"

namespace hyb {

template <typename T, int D, int F>
__global__ __launch_bounds__(kWave) void hyb_step_small_kernel(StepArgs a) {
  typedef Mma<T> M;
  typedef typename M::op_t op_t;
  typedef WaveFeatMap<T, D, F> WFM;
  constexpr int E = M::E, KW = M::KW, KD = D / KW, KL = kTile / KW, NS = D / kTile;
  constexpr int NT = F / kTile, NPAIR = 2 * NT;
  constexpr int f = 2 * F;

  const int lane = threadIdx.x, li = lane & 31, hh = lane >> 5;
  // Every kernel argument in one round of scalar loads: fetched where each
  // is first used, the later fields would wait behind the earlier ones, one
  // round trip each, before the first global load could issue.
  asm volatile("" ::"s"(a.s.B), "s"(a.s.Hq), "s"(a.s.Hkv), "s"(a.s.D), "s"(a.s.L), "s"(a.s.F), "s"(a.s.dtype),
               "s"(a.s.n_slots), "s"(a.s.out_f32),
               "s"(a.slots), "s"(a.block_len), "s"(a.out), "s"(a.alpha));
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L;
  // units (b, h, s): the slices of a head, then the heads of a KV group,
  // are neighbours (one XCD, one L2 for the Q, K, V and W rows they share)
  const int u = xcd_unit(blockIdx.x, a.s.B * Hq * NS);
  const int s = u % NS, bh = u / NS, b = bh / Hq, h = bh % Hq, g = h / (Hq / Hkv);
  // the slot and the block length, both requested before either is waited for
  int slot_v = b, lb_v = L;
  if (a.slots) slot_v = a.slots[b];
  if (a.block_len) lb_v = min(max(a.block_len[b], 0), L);
  const int slot = __builtin_amdgcn_readfirstlane(slot_v);
  const bool slot_ok = slot >= 0 && slot < a.s.n_slots;
  const int Lb = __builtin_amdgcn_readfirstlane(lb_v);
  if (Lb == 0) return;  // nothing to answer (uniform per wave)
  const int Lc = Lb - 1;
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
  const T* qb = (const T*)a.q + ((size_t)b * L * Hq + h) * D;
  const T* kb = (const T*)a.k + ((size_t)b * L * Hkv + g) * D;
  const T* vb = (const T*)a.v + ((size_t)b * L * Hkv + g) * D;
  const int c0 = s * kTile;
  const bool row_ok = li < Lb;

  // 1. Block operands (rows past Lb read row Lb-1, in bounds, then zeroed),
  //    then the state slice, so the block math can start while the state
  //    is in flight.  The loads are issued in the order of their first use
  //    (loads return in order) and, on the bf16 path, number fewer than the
  //    63 a wave can have outstanding, so that none of them waits for an
  //    earlier one to return before it can issue: V and z arrive as whole
  //    rows (two and one loads per lane) and are put into operand order
  //    through LDS.
  // (padding rows and keys are masked after every load has been issued: a
  // select next to its load would make the wave wait for it there)
  op_t qop[KD], kop[KD], vop[KL];
  {
    const T* qrow = qb + (size_t)min(li, Lc) * qstride + hh * E;
    const T* krow = kb + (size_t)min(li, Lc) * kstride + hh * E;
#pragma unroll
    for (int ks = 0; ks < KD; ++ks) {
      qop[ks] = load_op<T>(qrow + ks * KW);
      kop[ks] = load_op<T>(krow + ks * KW);
    }
  }
  op_t wop[NT][KD];
  WFM::load_w((const T*)a.W + (size_t)h * F * D, li, hh, wop);
  // V rows: on bf16, key (lane / 4) + 16 j, columns c0 + 8 (lane % 4) + 0..7
  // (rows past Lb read row Lb-1); on fp32 the V^T operand is gathered
  // directly (column c0 + li at keys row_of(ks, hh))
  constexpr int VR = E == 1 ? 1 : 2;
  bf16x8 vraw[VR];
  if constexpr (E == 1) {
    const T* vcol = vb + c0 + li;
#pragma unroll
    for (int ks = 0; ks < KL; ++ks) vop[ks] = vcol[(size_t)min(row_of(ks, hh), Lc) * kstride];
  } else {
#pragma unroll
    for (int j = 0; j < VR; ++j)
      vraw[j] = *reinterpret_cast<const bf16x8*>(vb + (size_t)min((lane >> 2) + 16 * j, Lc) * kstride + c0 +
                                                 8 * (lane & 3));
  }
  // State slice: column c0 + li of S_h (row c0 + li of the stored S_h^T),
  // features in the order of the phi registers (32p + row_of(ks*E + e, hh)
  // for k-step p*KL + ks); an out-of-range slot reads slot 0 (its outputs
  // are NaN).
  const size_t sbase = (size_t)(slot_ok ? slot : 0) * Hq + h;
  const float* __restrict__ srow = a.S + (sbase * D + c0 + li) * f;
  const float* __restrict__ zh = a.z + sbase * f;
  // z: f/64 consecutive values per lane (put into the order of the phi
  // registers through LDS), ahead of the state, which is needed last
  constexpr int ZPL = f / kWave;
  static_assert(ZPL == 1 || ZPL == 2 || ZPL == 4, "z is loaded as 1, 2 or 4 values per lane");
  float zv[ZPL];
  if constexpr (ZPL == 4) {
    const f32x4 t = *reinterpret_cast<const f32x4*>(zh + 4 * lane);
#pragma unroll
    for (int e = 0; e < 4; ++e) zv[e] = t[e];
  } else if constexpr (ZPL == 2) {
    const float2 t = *reinterpret_cast<const float2*>(zh + 2 * lane);
    zv[0] = t.x;
    zv[1] = t.y;
  } else {
    zv[0] = zh[lane];
  }
  constexpr int NKF = f / KW;  // k-steps over the features
  float sv[NKF][E];
#pragma unroll
  for (int kf = 0; kf < NKF; ++kf) {
    const int p = kf / KL, ks = kf % KL;
    if constexpr (E == 1) {
      sv[kf][0] = srow[p * kTile + row_of(ks, hh)];
    } else {
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(srow + p * kTile + row_of(ks * E, hh));
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(srow + p * kTile + row_of(ks * E + 4, hh));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sv[kf][e] = x0[e];
        sv[kf][4 + e] = x1[e];
      }
    }
  }

  const float alpha_h = a.alpha[h];  // the gate logit
  // Every load is issued here, ahead of the block math: moved to their uses
  // (as the compiler would) the state and z loads would wait behind it, a
  // second round trip to memory.
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int ks = 0; ks < KD; ++ks) {
    qop[ks] = keep_if<T>(row_ok, qop[ks]);
    kop[ks] = keep_if<T>(row_ok, kop[ks]);
  }
  if constexpr (E == 1) {
#pragma unroll
    for (int ks = 0; ks < KL; ++ks)
      if (row_of(ks, hh) >= Lb) vop[ks] = 0.0f;
  }

  // 2. Scores of query li against the block keys (keys in rows), softmax.
  const float scale = 1.0f / sqrtf((float)D);
  f32x16 sc = {};
#pragma unroll
  for (int ks = 0; ks < KD; ++ks) sc = M::mma(kop[ks], qop[ks], sc);
  float p[16];
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    p[i] = row_of(i, hh) < Lb ? sc[i] * scale : -INFINITY;
    m = fmaxf(m, p[i]);
  }
  m = fmaxf(m, xor32(m));
  float den = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    p[i] = row_of(i, hh) < Lb ? fast_exp(p[i] - m) : 0.0f;
    den += p[i];
  }
  den += xor32(den);

  // V^T of the slice ([column][key], rows padded against bank conflicts)
  // and z through LDS, read back in operand order.  (One wave per
  // workgroup: the barrier only orders the LDS accesses.)
  __shared__ float zs[f];
  __shared__ T vt[kTile][kTile + 4];
#pragma unroll
  for (int e = 0; e < ZPL; ++e) zs[ZPL * lane + e] = zv[e];
  if constexpr (E != 1) {
#pragma unroll
    for (int j = 0; j < VR; ++j)
#pragma unroll
      for (int c = 0; c < 8; ++c) vt[8 * (lane & 3) + c][(lane >> 2) + 16 * j] = vraw[j][c];
  }
  __syncthreads();
  f32x4 zr[NPAIR][4];
#pragma unroll
  for (int pp = 0; pp < NPAIR; ++pp)
#pragma unroll
    for (int j = 0; j < 4; ++j) zr[pp][j] = *reinterpret_cast<const f32x4*>(&zs[pp * kTile + row_of(4 * j, hh)]);
  if constexpr (E != 1) {
#pragma unroll
    for (int ks = 0; ks < KL; ++ks) {
      vop[ks] = lds_op_perm<T>(&vt[li][0], ks, hh, 0);
#pragma unroll
      for (int e = 0; e < E; ++e)
        if (row_of(ks * E + e, hh) >= Lb) vop[ks][e] = (T)0.0f;
    }
  }

  // 3. phi(q_li) and lin_den = phi(q_li) . z.
  float phi[NPAIR][16];
  WFM::compute(wop, qop, phi, row_ok);
  float lz = 0.0f;
#pragma unroll
  for (int pp = 0; pp < NPAIR; ++pp)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) lz += phi[pp][4 * j + e] * zr[pp][j][e];
  lz += xor32(lz);

  // 4. Merge coefficients (overflow-safe form): out = ca a' + cb r with
  //    a' = P V relative to the row maximum and r = phi(Q) S.
  const float lw = log_sigmoid(alpha_h);
  float ca, cb;
  if (lz > 0.0f) {
    const float la = lw + m, lb = logf(lz);
    const float c = fmaxf(la, lb);
    const float ea = expf(la - c), eb = expf(lb - c);
    const float inv = 1.0f / (ea * den + eb);
    ca = ea * inv;
    cb = eb * inv / lz;
  } else {
    ca = 1.0f / den;
    cb = 0.0f;
  }
  if (!slot_ok) ca = cb = __builtin_nanf("");

  // 5. The slice's products: rows c0 + row_of(i, hh), column (query) li.
  f32x16 apv = {}, rd = {};
#pragma unroll
  for (int ks = 0; ks < KL; ++ks) apv = mma_split_b<T>(vop[ks], &p[ks * E], apv);
#pragma unroll
  for (int kf = 0; kf < NKF; ++kf) {
    const int pp = kf / KL, ks = kf % KL;
    rd = M::mma(cvt_op<T>(sv[kf]), cvt_op<T>(&phi[pp][ks * E]), rd);
  }

  // 6. Outputs of query li (4 consecutive columns per run).
  if (!row_ok) return;
  const size_t ob = (((size_t)b * L + li) * Hq + h) * D + c0;
#pragma unroll
  for (int j = 0; j < 16; j += 4) {
    float o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = ca * apv[j + e] + cb * rd[j + e];
    store_out4<T>(a.out, ob + row_of(j, hh), o, a.s.out_f32);
  }
}

template <typename T, int D, int F>
static hipError_t small_go(const StepArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((hyb_step_small_kernel<T, D, F>), dim3(a.s.B * a.s.Hq * (D / kTile)),
                     dim3(kWave), 0, st, a);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t small_f(const StepArgs& a, hipStream_t st) {
  switch (a.s.F) {
    case 32: return small_go<T, D, 32>(a, st);
    case 64: return small_go<T, D, 64>(a, st);
    case 128: return small_go<T, D, 128>(a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_step_small(const StepArgs& a, hipStream_t st) {
  if (a.s.dtype == 1)
    return a.s.D == 64 ? small_f<bf16, 64>(a, st) : small_f<bf16, 128>(a, st);
  return a.s.D == 64 ? small_f<float, 64>(a, st) : small_f<float, 128>(a, st);
}

}  // namespace hyb
