// prefill.hip -- block-causal prefill of a prompt into the recurrent state
// (Figure 2 pattern): block c is answered against the state of blocks
// 0..c-1 -- exact softmax inside the block, linear readout of the state,
// gated merge (Section 3.1) -- and is then committed,
// S += phi(K_c)^T V_c, z += sum phi(K_c).
//
// Sequence segments.  The prompt's blocks are cut into nseg segments so that
// the grid fills the chip.  A first launch (delta mode) computes each
// segment's own state increment dS_s = sum_{c in s} phi(K_c)^T V_c and dz_s
// into the caller's workspace (the last segment's is not needed); the second
// launch (walk mode) starts segment s from S + sum_{s' < s} dS_s' and walks
// its blocks as below; the last segment writes the final state.  Only the
// associativity of the sum is used, so the result is the sequential one up to
// rounding order.  Without outputs, only the last segment walks.
//
// Within a segment, one workgroup per (request b, query head h) walks the
// blocks in order, with the next block's Q, K and V in flight while the
// current one is computed.
// Wave w of NW = D/32 keeps state columns 32w .. 32w+31 of all f rows in fp32
// MFMA accumulators for the whole prompt, so the state is read from HBM once
// and written once.  The accumulator tile doubles as the A operand of the
// readout O_lin^T = S^T phi(Q)^T: register j of the flattened tile is
// contraction element j % E of k-step j / E, i.e. state row
// r = 32*(j/16) + row_of(j%16, hh), and phi(Q) is read from LDS in that
// order.  Block tokens enter every product in the accumulator order of the
// score tile (token row_of(ks*E+e, hh)), so one set of V registers serves
// both P V and the commit.  As in the commit kernel, phi(K) enters the state
// update as a bf16 pair hi + lo on the bf16 path.
#include "device.h"
#include "featmap.h"
#include "launch.h"

namespace hyb {

template <typename T, int D, int F>
struct PrefillCfg {
  typedef Mma<T> M;
  typedef typename M::op_t op_t;
  static constexpr int NW = D / kTile;
  static constexpr int f = 2 * F;
  static constexpr int NRT = f / kTile;
  static constexpr int KD = D / M::KW;
  static constexpr int KF = f / M::KW;
  static constexpr int KL = kTile / M::KW;
  static constexpr int PHI_LD = f + 16 / (int)sizeof(T);
  static constexpr int PT_LD = kTile + 16 / (int)sizeof(T);
  static constexpr int NPART = sizeof(T) == 2 ? 2 : 1;  // hi (+ lo) parts
  typedef FeatMap<T, D, F, NW> FM;
  struct alignas(16) Smem {
    T phiQ[kTile][PHI_LD];         // phi(q_i)[r] at [i][r]
    T phiKT[NPART][f][PT_LD];      // phi(k_t)[r] at [part][r][t]
    float z[f];
    float lden[NW][kTile];         // per-wave partial phi(q_i) . z
    typename FM::Smem fq, fk;
  };
};

template <typename T, int D, int F>
__global__ __launch_bounds__(kWave*(D / kTile)) void hyb_prefill_kernel(
    PrefillArgs a, int nseg, int seg_blocks, int delta) {
  typedef PrefillCfg<T, D, F> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  typedef typename C::FM FM;
  constexpr int f = C::f, E = M::E, KW = M::KW;
  __shared__ typename C::Smem sh;

  const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L, T_ = a.T;
  // Unit u = (b, h) varies fastest, so the heads of one KV group and segment
  // are neighbours (on one XCD) and share K and V in L2.
  const int units = a.s.B * Hq, nseg_here = delta ? nseg - 1 : nseg;
  const int vix = xcd_unit(blockIdx.x, units * nseg_here);
  const int u = vix % units, seg = vix / units;
  const int b = u / Hq, h = u % Hq, g = h / (Hq / Hkv);
  const int slot = a.slots ? a.slots[b] : b;
  const bool want_out = !delta && a.out != nullptr;
  const bool last = seg == nseg - 1;
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
  const int col = w * kTile + li;
  const int nblk = T_ / L;
  const int blk0 = seg * seg_blocks, blk1 = min(nblk, blk0 + seg_blocks);
  if (!delta && !want_out && !last) return;  // state only: the last segment walks
  if (slot < 0 || slot >= a.s.n_slots) {  // uniform per workgroup
    if (want_out) {
      const size_t ob = ((size_t)b * T_ * Hq + h) * D;
      for (int t = blk0 * L; t < blk1 * L; ++t)
        for (int c = tid; c < D; c += blockDim.x)
          store_out1<T>(a.out, ob + (size_t)t * qstride + c, __builtin_nanf(""),
                        a.s.out_f32);
    }
    return;
  }
  const size_t sbase = (size_t)slot * Hq + h;
  float* __restrict__ Sh = a.S + sbase * f * D;
  float* __restrict__ zh = a.z + sbase * f;
  // Workspace: dS [units][nseg-1][D][f] (transposed, as S), then dz
  // [units][nseg-1][f].
  float* __restrict__ wsS = a.ws + (size_t)u * (nseg - 1) * D * f;
  float* __restrict__ wsz = a.ws + (size_t)units * (nseg - 1) * D * f + (size_t)u * (nseg - 1) * f;

  // Starting state: zero for a delta, else S plus the earlier segments'
  // increments, all in the accumulator layout.
  f32x16 sacc[C::NRT];
  auto add_state = [&](const float* src, bool first) {
#pragma unroll
    for (int rt = 0; rt < C::NRT; ++rt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {  // rows rt*32 + j*8 + hh*4 .. +3: 16 bytes
        const f32x4 x = *reinterpret_cast<const f32x4*>(
            src + (size_t)col * f + rt * kTile + row_of(4 * j, hh));
#pragma unroll
        for (int r = 0; r < 4; ++r) sacc[rt][4 * j + r] = first ? x[r] : sacc[rt][4 * j + r] + x[r];
      }
  };
  if (delta) {
#pragma unroll
    for (int rt = 0; rt < C::NRT; ++rt) sacc[rt] = f32x16{};
    for (int r = tid; r < f; r += blockDim.x) sh.z[r] = 0.0f;
  } else {
    add_state(Sh, true);
    for (int s = 0; s < seg; ++s) add_state(wsS + (size_t)s * D * f, false);
    for (int r = tid; r < f; r += blockDim.x) {
      float zr = zh[r];
      for (int s = 0; s < seg; ++s) zr += wsz[(size_t)s * f + r];
      sh.z[r] = zr;
    }
  }

  const T* __restrict__ Wt_h = (const T*)a.W + (size_t)h * F * D;
  op_t wop[FM::PPW][C::KD];  // W_h^T operands, kept for the whole prompt
  FM::load_w(Wt_h, w, li, hh, wop);
  const float scale = 1.0f / sqrtf((float)D);
  const float lw = want_out ? log_sigmoid(a.alpha[h]) : 0.0f;
  const bool row_ok = li < L;
  const int lrow = min(li, L - 1);

  // Block operands.  Unconditional, in-bounds loads: padding rows read row
  // L-1 and are zeroed by a select later; the prefetch past the segment's
  // last block re-reads that block.
  auto load_block = [&](int blk, op_t (&ko)[C::KD], op_t (&qo)[C::KD],
                        op_t (&vo)[C::KL]) {
    const size_t t0 = (size_t)blk * L;
    const T* kb = (const T*)a.k + (((size_t)b * T_ + t0) * Hkv + g) * D;
    const T* vb = (const T*)a.v + (((size_t)b * T_ + t0) * Hkv + g) * D;
    const T* krow = kb + (size_t)lrow * kstride + hh * E;
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks) ko[ks] = load_op<T>(krow + ks * KW);
#pragma unroll
    for (int ks = 0; ks < C::KL; ++ks)
      vo[ks] = load_rows_op<T>(vb + col, kstride, ks, hh, L, false);
    if (want_out) {
      const T* qrow = (const T*)a.q + (((size_t)b * T_ + t0) * Hq + h) * D +
                      (size_t)lrow * qstride + hh * E;
#pragma unroll
      for (int ks = 0; ks < C::KD; ++ks) qo[ks] = load_op<T>(qrow + ks * KW);
    }
  };
  op_t kop[C::KD], qop[C::KD], vop[C::KL];
#pragma unroll
  for (int ks = 0; ks < C::KD; ++ks) qop[ks] = M::zero();
  if (blk0 < blk1) load_block(blk0, kop, qop, vop);

  for (int blk = blk0; blk < blk1; ++blk) {
    const size_t t0 = (size_t)blk * L;
    op_t kn[C::KD], qn[C::KD], vn[C::KL];
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks) qn[ks] = M::zero();
    load_block(min(blk + 1, blk1 - 1), kn, qn, vn);
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks) {
      kop[ks] = keep_if<T>(row_ok, kop[ks]);
      qop[ks] = keep_if<T>(row_ok, qop[ks]);
    }

    lds_barrier();  // previous block's LDS readers are done
    float vk[FM::PPW][16], vq[FM::PPW][16];
    FM::logits(wop, kop, w, li, hh, vk, sh.fk);
    if (want_out) FM::logits(wop, qop, w, li, hh, vq, sh.fq);

    // In-block softmax branch (keys in rows, queries in columns).
    f32x16 acc_sm = {};
    float m = 0.0f, den = 1.0f;
    if (want_out) {
      f32x16 sc = {};
#pragma unroll
      for (int ks = 0; ks < C::KD; ++ks) sc = M::mma(kop[ks], qop[ks], sc);
      float p[16];
      m = -INFINITY;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        p[i] = row_of(i, hh) < L ? sc[i] * scale : -INFINITY;
        m = fmaxf(m, p[i]);
      }
      m = fmaxf(m, xor32(m));
      den = 0.0f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        p[i] = row_of(i, hh) < L ? fast_exp(p[i] - m) : 0.0f;
        den += p[i];
      }
      den += xor32(den);
#pragma unroll
      for (int ks = 0; ks < C::KL; ++ks)
        acc_sm = mma_split_b<T>(vop[ks], &p[ks * E], acc_sm);
    }

    lds_barrier();
    FM::exps(w, li, hh, vk, sh.fk);
    if (want_out) FM::exps(w, li, hh, vq, sh.fq);
    lds_barrier();
    FM::normalise(w, li, hh, vk, sh.fk, [&](int f0, const float* x4) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = row_ok ? x4[e] : 0.0f;
        const T hi = from_f32<T>(x);
        sh.phiKT[0][f0 + e][li] = hi;
        if constexpr (C::NPART == 2)
          sh.phiKT[1][f0 + e][li] = from_f32<T>(x - to_f32(hi));
      }
    });
    if (want_out) {
      // phi(q) to LDS and this wave's part of lin_den = phi(q) . z (the
      // features of the pairs it owns), summed over the waves below.
      float lz = 0.0f;
      FM::normalise(w, li, hh, vq, sh.fq, [&](int f0, const float* x4) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          sh.phiQ[li][f0 + e] = from_f32<T>(x4[e]);
          lz += x4[e] * sh.z[f0 + e];
        }
      });
      lz += xor32(lz);
      if (hh == 0) sh.lden[w][li] = lz;
    }
    lds_barrier();

    if (want_out) {
      // Readout against the state of the blocks before this one.
      f32x16 acc_lin = {};
      float lden = 0.0f;
#pragma unroll
      for (int ww = 0; ww < C::NW; ++ww) lden += sh.lden[ww][li];
#pragma unroll
      for (int ks = 0; ks < C::KF; ++ks) {
        const op_t pb = lds_op_perm<T>(&sh.phiQ[li][0], ks, hh, 0);
        op_t sa;
        if constexpr (E == 1) {
          sa = sacc[ks / 16][ks % 16];
        } else {
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const int j = ks * E + e;  // flattened accumulator register
            sa[e] = (T)sacc[j / 16][j % 16];
          }
        }
        acc_lin = M::mma(sa, pb, acc_lin);
      }
      if (row_ok) {
        float ca = 1.0f, cz = 0.0f, rz = 0.0f;
        if (lden > 0.0f) {
          const float la = lw + m, lb = logf(lden);
          const float c = fmaxf(la, lb);
          ca = expf(la - c);
          cz = expf(lb - c);
          rz = 1.0f / lden;
        }
        const float inv = 1.0f / (ca * den + cz);
        const size_t obase = (((size_t)b * T_ + t0 + li) * Hq + h) * D;
#pragma unroll
        for (int i = 0; i < 16; i += 4) {
          float o[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            o[e] = (ca * acc_sm[i + e] + cz * (acc_lin[i + e] * rz)) * inv;
          store_out4<T>(a.out, obase + w * kTile + row_of(i, hh), o, a.s.out_f32);
        }
      }
    }

    // Commit the block: S += phi(K)^T V in the accumulators.
#pragma unroll
    for (int rt = 0; rt < C::NRT; ++rt)
#pragma unroll
      for (int ks = 0; ks < C::KL; ++ks)
#pragma unroll
        for (int part = 0; part < C::NPART; ++part)
          sacc[rt] = M::mma(
              lds_op_perm<T>(&sh.phiKT[part][rt * kTile + li][0], ks, hh, 0),
              vop[ks], sacc[rt]);
    lds_barrier();  // every wave has read z for this block
    // z += sum_t phi(k_t): row r of phiKT holds the 32 tokens contiguously
    // (zero past the block length), read 16 bytes at a time.
    for (int r = tid; r < f; r += blockDim.x) {
      float s = 0.0f;
#pragma unroll
      for (int part = 0; part < C::NPART; ++part)
#pragma unroll
        for (int t0 = 0; t0 < kTile; t0 += 16 / (int)sizeof(T)) {
          const uint4 x = *reinterpret_cast<const uint4*>(&sh.phiKT[part][r][t0]);
          const T* xt = reinterpret_cast<const T*>(&x);
#pragma unroll
          for (int e = 0; e < 16 / (int)sizeof(T); ++e) s += to_f32(xt[e]);
        }
      sh.z[r] += s;
    }
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks) {
      kop[ks] = kn[ks];
      qop[ks] = qn[ks];
    }
#pragma unroll
    for (int ks = 0; ks < C::KL; ++ks) vop[ks] = vn[ks];
  }

  // A delta goes to the workspace; the last segment's walk writes the state.
  if (!delta && !last) return;
  float* dstS = delta ? wsS + (size_t)seg * D * f : Sh;
  float* dstz = delta ? wsz + (size_t)seg * f : zh;
#pragma unroll
  for (int rt = 0; rt < C::NRT; ++rt)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<f32x4*>(dstS + (size_t)col * f + rt * kTile + row_of(4 * j, hh)) =
          f32x4{sacc[rt][4 * j], sacc[rt][4 * j + 1], sacc[rt][4 * j + 2], sacc[rt][4 * j + 3]};
  lds_barrier();
  for (int r = tid; r < f; r += blockDim.x) dstz[r] = sh.z[r];
}

template <typename T, int D, int F>
static hipError_t prefill_go(const PrefillArgs& a, hipStream_t st) {
  const int units = a.s.B * a.s.Hq, nblk = a.T / a.s.L;
  const int nseg = prefill_segments(a.s, a.T);
  const int seg_blocks = (nblk + nseg - 1) / nseg;
  const dim3 block(kWave * (D / kTile));
  if (nseg > 1) {
    hipLaunchKernelGGL((hyb_prefill_kernel<T, D, F>), dim3(units * (nseg - 1)), block, 0, st,
                       a, nseg, seg_blocks, 1);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((hyb_prefill_kernel<T, D, F>), dim3(units * nseg), block, 0, st, a, nseg,
                     seg_blocks, 0);
  return hipGetLastError();
}

template <typename T, int D, int F>
static hipError_t prefill_delta_go(const PrefillArgs& a, hipStream_t st) {
  const int units = a.s.B * a.s.Hq, nblk = a.T / a.s.L;
  const int nseg = prefill_segments(a.s, a.T);
  const int seg_blocks = (nblk + nseg - 1) / nseg;
  if (nseg <= 1) return hipSuccess;
  hipLaunchKernelGGL((hyb_prefill_kernel<T, D, F>), dim3(units * (nseg - 1)),
                     dim3(kWave * (D / kTile)), 0, st, a, nseg, seg_blocks, 1);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t prefill_delta_f(const PrefillArgs& a, hipStream_t st) {
  switch (a.s.F) {
    case 32: return prefill_delta_go<T, D, 32>(a, st);
    case 64: return prefill_delta_go<T, D, 64>(a, st);
    case 128: return prefill_delta_go<T, D, 128>(a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_prefill_delta(const PrefillArgs& a, hipStream_t st) {
  if (a.s.dtype == 1)
    return a.s.D == 64 ? prefill_delta_f<bf16, 64>(a, st) : prefill_delta_f<bf16, 128>(a, st);
  return a.s.D == 64 ? prefill_delta_f<float, 64>(a, st) : prefill_delta_f<float, 128>(a, st);
}

// Segments: enough (request, head, segment) workgroups to cover the chip
// about twice, at most 8 segments (the walk of segment s reads the s earlier
// increments) and at least 4 blocks per segment.
int prefill_segments(const Shape& s, int T) {
  const int units = s.B * s.Hq, nblk = T / s.L;
  int nseg = (512 + units - 1) / units;
  if (nseg > 8) nseg = 8;
  if (nseg > nblk / 4) nseg = nblk / 4;
  if (nseg < 1) nseg = 1;
  // Every segment must own at least one block at the rounded-up length.
  for (; nseg > 1; --nseg)
    if ((nseg - 1) * ((nblk + nseg - 1) / nseg) < nblk) break;
  return nseg;
}

size_t prefill_ws_bytes(const Shape& s, int T) {
  const int nseg = prefill_segments(s, T);
  if (nseg <= 1) return 0;
  const size_t f = 2 * (size_t)s.F;
  return (size_t)s.B * s.Hq * (nseg - 1) * ((size_t)s.D * f + f) * 4;
}

template <typename T, int D>
static hipError_t prefill_f(const PrefillArgs& a, hipStream_t st) {
  switch (a.s.F) {
    case 32: return prefill_go<T, D, 32>(a, st);
    case 64: return prefill_go<T, D, 64>(a, st);
    case 128: return prefill_go<T, D, 128>(a, st);
  }
  return hipErrorInvalidValue;
}

template <typename T>
static hipError_t prefill_d(const PrefillArgs& a, hipStream_t st) {
  switch (a.s.D) {
    case 64: return prefill_f<T, 64>(a, st);
    case 128: return prefill_f<T, 128>(a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_prefill(const PrefillArgs& a, hipStream_t st) {
  return a.s.dtype == 1 ? prefill_d<bf16>(a, st) : prefill_d<float>(a, st);
}

}  // namespace hyb
