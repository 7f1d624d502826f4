// backward.hip -- gradient of the block-causal hybrid layer with respect to
// its feature-map weights W and gate logits alpha: the attention transfer of
// Section 3.2 (Stage 1), whose only trainable parameters are {W, alpha}.
//
// Forward (Figure 2 pattern, from an empty state): block c of the sequence
// is answered against S_{c-1}, z_{c-1} (exact softmax inside the block,
// linear readout, shared-normaliser merge of Section 3.1) and then committed.
// With g = dL/dout, N = w sm_num + lin_num, D = w sm_den + lin_den:
//   dL/dN_i = g_i / D_i,  dL/dD_i = -(g_i . out_i) / D_i
//   dL/dw  += dL/dN_i . sm_num_i + dL/dD_i sm_den_i
//   dL/dphi(q_i) = S_{c-1} dL/dN_i + z_{c-1} dL/dD_i
//   dL/dphi(k_t) = Gbar_c v_t + gz_c,  Gbar_c = sum over the queries of the
//                  blocks after c of phi(q_i) dL/dN_i^T (gz_c likewise)
//   feature map: dL/du_j = p_j (dp_j - <dp,p>) - n_j (dn_j - <dn,n>),
//                dL/dW[:, j] += x dL/du_j.
// In attention-transfer mode g_i = 2 (out_i - target_i) is formed in
// registers from the teacher's output; out itself never reaches memory.
//
// Kernels (one workgroup per (request, head, sequence segment), NW = D/32
// waves; segments as in the prefill, so the grid fills the chip):
//   1. the prefill's delta launch: each segment's state increment;
//   2. forward walk: per block out, dL/dN, dL/dD, dL/dphi(Q) and the query
//      part of dL/dW and dL/dalpha; dL/dN^T and dL/dD go to the workspace.
//      On the bf16 path hyb_bwd_fpipe_kernel (pipelined, below) keeps S and
//      S^T both in fp32 accumulators; on fp32 hyb_bwd_fwd_kernel keeps S
//      columns 32w..+31 in accumulators (the readout operand, as in the
//      prefill) and copies S_{c-1} to LDS each block as [feature][column]
//      operands for dL/dphi(Q), which contracts over the head dimension;
//   3. each segment's sum of phi(Q)^T dL/dN (and phi(Q)^T dL/dD):
//      hyb_bwd_gdelta_kernel on the bf16 path (pipelined, below),
//      hyb_bwd_rev_kernel in delta mode on fp32;
//   4. reverse walk with Gbar^T in the accumulators, the key part of dL/dW:
//      hyb_bwd_rwalk_kernel on the bf16 path (pipelined, below),
//      hyb_bwd_rev_kernel in walk mode on fp32;
//   5. hyb_bwd_reduce_kernel: sums the per-(request, segment) partials in a
//      fixed order (bitwise reproducible, no atomics).
// On the bf16 path phi(K), phi(Q) (as an update operand) and dL/du enter the
// matrix products as bf16 pairs hi + lo; the state, Gbar and dL/dN as bf16.
#include <type_traits>

#include "device.h"
#include "featmap.h"
#include "launch.h"

namespace hyb {

template <typename T, int D, int F>
struct BwdCfg {
  typedef Mma<T> M;
  typedef typename M::op_t op_t;
  static constexpr int NW = D / kTile;      // waves = 32-column slices of d
  static constexpr int f = 2 * F;
  static constexpr int NRT = f / kTile;     // 32-feature tiles
  static constexpr int NT = F / kTile;      // tiles per sign
  static constexpr int RPW = (NRT + NW - 1) / NW;  // feature tiles per wave
  static constexpr int KD = D / M::KW;
  static constexpr int KL = kTile / M::KW;
  static constexpr int NPART = sizeof(T) == 2 ? 2 : 1;
  static constexpr int PAD = 16 / (int)sizeof(T);
  typedef FeatMap<T, D, F, NW> FM;
  static_assert(FM::PPW == RPW, "one feature-map pair per feature tile");
  struct alignas(16) SmemF {
    T st[NPART][f][D + PAD];             // S_{c-1} as operands, [part][r][c]
    T phiQ[NPART][kTile][f + PAD];       // phi(q_i)[r] at [part][i][r]
    T phiKT[NPART][f][kTile + PAD];      // phi(k_t)[r] at [part][r][t]
    T gn[NPART][kTile][D + PAD];         // dL/dN_i[c] at [part][i][c]
    T duT[2][NPART][F][kTile + PAD];     // +-dL/du from each sign, [j][i]
    float z[f];
    float lden[NW][kTile];
    float red[NW][kTile][2];
    float jsum[NRT][kTile];
    float gd[kTile];
    float fin[NW][2];
    typename FM::Smem fq, fk;
  };
  struct alignas(16) SmemB {
    T phiQT[NPART][f][kTile + PAD];      // phi(q_i)[r] at [part][r][i]
    T duT[2][NPART][F][kTile + PAD];
    float gz[f];
    float jsum[NRT][kTile];
    float gd[kTile];
    typename FM::Smem fq, fk;
  };
};

// Workspace layout (floats unless noted), every part 256-byte aligned:
//   prefill deltas dS [units][nseg-1][D][f], dz [units][nseg-1][f]
//   Gbar deltas   dG [units][nseg][D][f] (transposed like S), dgz [units][nseg][f]
//   dL/dN^T        gnT [units][nblk][D][32]
//   dL/dD          gd  [units][nblk][32]
//   partial dW     dwq, dwk [units][nseg][F][D]
//   partial scalars red [units][nseg][2]  (dL/dalpha, loss)
// and, when the input gradients are formed:
//   dL/du of the queries   duq [units][T][F]
//   dL/du of the keys      duk [units][T][F]
//   Gbar_c^T phi(k_t)       dvl [units][T][D]  (the state part of dL/dv_t)
struct BwdLayout {
  size_t dS, dG, dgz, gnT, gd, dwq, dwk, red, duq, duk, dvl, total;
};

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

static BwdLayout bwd_layout(const Shape& s, int T, bool inputs) {
  const size_t units = (size_t)s.B * s.Hq, f = 2 * (size_t)s.F;
  const SegPlan plan = segment_plan(s, T);
  const int nseg = plan.nseg, nblk = T / s.L;
  const size_t npc = plan.npieces() > 0 ? plan.npieces() : 1;
  BwdLayout l;
  size_t o = 0;
  l.dS = o;
  o = align256(o + prefill_delta_ws_bytes(s, plan));
  l.dG = o;
  o = align256(o + units * npc * s.D * f * 4);
  l.dgz = o;
  o = align256(o + units * npc * f * 4);
  l.gnT = o;
  o = align256(o + units * nblk * s.D * kTile * 4);
  l.gd = o;
  o = align256(o + units * nblk * kTile * 4);
  l.dwq = o;
  o = align256(o + units * nseg * s.F * s.D * 4);
  l.dwk = o;
  o = align256(o + units * nseg * s.F * s.D * 4);
  l.red = o;
  o = align256(o + units * nseg * 2 * 4);
  l.duq = l.duk = l.dvl = o;
  if (inputs) {
    l.duq = o;
    o = align256(o + units * T * s.F * 4);
    l.duk = o;
    o = align256(o + units * T * s.F * 4);
    l.dvl = o;
    o = align256(o + units * T * s.D * 4);
  }
  l.total = o;
  return l;
}

size_t backward_ws_bytes(const Shape& s, int T, bool inputs) {
  return bwd_layout(s, T, inputs).total;
}

struct BwdKArgs {
  BackwardArgs a;
  int nseg, seg_blocks, nblk;
  // The increments come in pieces of at most pb blocks, ppseg per segment,
  // npc in all.  State increments: pieces of segments 0 .. nseg-2, dS
  // [units][npc][D][f] and dz [units][npc][f]; the forward walk of segment s
  // starts from the sum of pieces 0 .. s*ppseg - 1.  Reverse increments:
  // pieces of segments 1 .. nseg-1 (rev_piece), dG [units][npc][D][f] and
  // dgz [units][npc][f]; the reverse walk of segment s starts from the sum
  // of pieces s*ppseg .. npc - 1.
  int ppseg, npc, pb;
  float *dS, *dz, *dG, *dgz, *gd, *dwq, *dwk, *red, *gnT;
  float *duq, *duk, *dvl;  // input-gradient intermediates (null otherwise)
};

// Blocks blk0 .. blk1-1 of piece pc of the reverse increments (empty where
// the last segment is short).
__device__ inline void rev_piece(const BwdKArgs& ka, int pc, int& blk0, int& blk1) {
  const int seg = pc / ka.ppseg + 1, k = pc % ka.ppseg;
  blk0 = min(ka.nblk, seg * ka.seg_blocks + k * ka.pb);
  blk1 = max(blk0, min(ka.nblk, min(seg * ka.seg_blocks + (k + 1) * ka.pb, (seg + 1) * ka.seg_blocks)));
}

// LDS of the reverse walk's extra work when the input gradients are formed:
// Gbar^T of the blocks after this one and phi(K), as operands.
template <typename T, int D, int F>
struct RevInSmem {
  static constexpr int NPART = sizeof(T) == 2 ? 2 : 1;
  static constexpr int PAD = 16 / (int)sizeof(T);
  T gT[NPART][D][2 * F + PAD];      // Gbar^T[c][r]
  T phiK[NPART][kTile][2 * F + PAD];  // phi(k_t)[r] at [t][r]
};
struct NoSmem {
  char unused;
};

// Accumulator registers ks*E .. ks*E+E-1 of a tile as a T operand (the tile's
// rows become the contraction index, in row_of order).
template <typename T>
__device__ inline typename Mma<T>::op_t acc_op(const f32x16& x, int ks) {
  typedef Mma<T> M;
  typename M::op_t r;
  if constexpr (M::E == 1) {
    r = x[ks];
  } else {
#pragma unroll
    for (int e = 0; e < M::E; ++e) r[e] = (T)x[ks * M::E + e];
  }
  return r;
}

// The rounding remainders x - T(x) of the same registers: with acc_op they
// carry x as a pair hi + lo (about 16 significant bits on the bf16 path).
template <typename T>
__device__ inline typename Mma<T>::op_t acc_op_lo(const f32x16& x, int ks) {
  typedef Mma<T> M;
  typename M::op_t r;
  if constexpr (M::E == 1) {
    r = 0.0f;
  } else {
#pragma unroll
    for (int e = 0; e < M::E; ++e) {
      const float v = x[ks * M::E + e];
      r[e] = (T)(v - as_operand<T>(v));
    }
  }
  return r;
}

// acc_op and acc_op_lo of the same registers in one pass on the bf16 path:
// one paired rounding for two hi parts and one for two lo parts.
__device__ inline void acc_op_pair(const f32x16& x, int ks, bf16x8& hi, bf16x8& lo) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  u32x4 h4, l4;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float x0 = x[ks * 8 + 2 * e], x1 = x[ks * 8 + 2 * e + 1];
    const uint32_t h = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)x0, (__bf16)x1});
    const float h0 = __builtin_bit_cast(float, h << 16);
    const float h1 = __builtin_bit_cast(float, h & 0xffff0000u);
    h4[e] = h;
    l4[e] = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)(x0 - h0), (__bf16)(x1 - h1)});
  }
  hi = __builtin_bit_cast(bf16x8, h4);
  lo = __builtin_bit_cast(bf16x8, l4);
}

// E fp32 values from p as an operand pair hi + lo (lo is zero on fp32).
template <typename T>
__device__ inline void load_split_op(const float* p, typename Mma<T>::op_t& hi,
                                     typename Mma<T>::op_t& lo) {
  typedef Mma<T> M;
  if constexpr (M::E == 1) {
    hi = *p;
    lo = 0.0f;
  } else {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p);
    const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
    const float x[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      hi[e] = (T)x[e];
      lo[e] = (T)(x[e] - as_operand<T>(x[e]));
    }
  }
}

// Eight fp32 values (a, then b) as a bf16 operand pair hi + lo.
__device__ inline void split_op(const f32x4& a, const f32x4& b, bf16x8& hi, bf16x8& lo) {
  const float x[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    hi[e] = (bf16)x[e];
    lo[e] = (bf16)(x[e] - as_operand<bf16>(x[e]));
  }
}

// Wave-wide sum (64 lanes).
__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// ---------------------------------------------------------------------------
// 2. Forward walk.
// ---------------------------------------------------------------------------
template <typename T, int D, int F, bool IN>
__global__ __launch_bounds__(kWave*(D / kTile)) void hyb_bwd_fwd_kernel(BwdKArgs ka) {
  typedef BwdCfg<T, D, F> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  typedef typename C::FM FM;
  constexpr int f = C::f, E = M::E, KW = M::KW, NW = C::NW, RPW = C::RPW;
  constexpr int NT = C::NT, NRT = C::NRT;
  __shared__ typename C::SmemF sh;
  const BackwardArgs& a = ka.a;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);  // wave-uniform
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L, T_ = a.T;
  const int units = a.s.B * Hq, nseg = ka.nseg;
  const int vix = xcd_unit(blockIdx.x, units * nseg);
  const int u = vix % units, seg = vix / units;
  const int b = u / Hq, h = u % Hq, g = h / (Hq / Hkv);
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
  const int col = w * kTile + li;
  const int blk0 = seg * ka.seg_blocks, blk1 = min(ka.nblk, blk0 + ka.seg_blocks);
  const bool tmode = a.target != nullptr;

  // Starting state: the increments of the earlier segments (the sequence
  // starts from an empty state).
  f32x16 sacc[NRT];
#pragma unroll
  for (int rt = 0; rt < NRT; ++rt) sacc[rt] = f32x16{};
  for (int r = tid; r < f; r += blockDim.x) sh.z[r] = 0.0f;
  for (int pc = 0; pc < seg * ka.ppseg; ++pc) {
    const float* src = ka.dS + ((size_t)u * ka.npc + pc) * D * f;
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
      for (int i = 0; i < 16; ++i) sacc[rt][i] += src[(size_t)col * f + rt * kTile + row_of(i, hh)];
    const float* zs = ka.dz + ((size_t)u * ka.npc + pc) * f;
    for (int r = tid; r < f; r += blockDim.x) sh.z[r] += zs[r];
  }

  const T* __restrict__ Wt_h = (const T*)a.W + (size_t)h * F * D;
  op_t wop[FM::PPW][C::KD];
  FM::load_w(Wt_h, w, li, hh, wop);
  const float scale = 1.0f / sqrtf((float)D);
  const float lw = log_sigmoid(a.alpha[h]);
  const float one_minus_w = expf(log_sigmoid(-a.alpha[h]));
  const bool row_ok = li < L;
  const int lrow = min(li, L - 1);

  f32x16 dwacc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) dwacc[t] = f32x16{};
  float dal = 0.0f, lss = 0.0f;

  for (int blk = blk0; blk < blk1; ++blk) {
    const size_t t0 = (size_t)blk * L;
    const T* kb = (const T*)a.k + (((size_t)b * T_ + t0) * Hkv + g) * D;
    const T* vb = (const T*)a.v + (((size_t)b * T_ + t0) * Hkv + g) * D;
    const T* qb = (const T*)a.q + (((size_t)b * T_ + t0) * Hq + h) * D;
    op_t kop[C::KD], qop[C::KD], vop[C::KL];
    {
      const T* krow = kb + (size_t)lrow * kstride + hh * E;
      const T* qrow = qb + (size_t)lrow * qstride + hh * E;
#pragma unroll
      for (int ks = 0; ks < C::KD; ++ks) {
        kop[ks] = keep_if<T>(row_ok, load_op<T>(krow + ks * KW));
        qop[ks] = keep_if<T>(row_ok, load_op<T>(qrow + ks * KW));
      }
#pragma unroll
      for (int ks = 0; ks < C::KL; ++ks)
        vop[ks] = load_rows_op<T>(vb + col, kstride, ks, hh, L, false);
    }

    lds_barrier();  // the previous block's LDS readers are done
    // S_{c-1} to LDS as operands (hi + lo): column col of every feature row.
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const T hi = from_f32<T>(sacc[rt][i]);
        sh.st[0][rt * kTile + row_of(i, hh)][col] = hi;
        if constexpr (C::NPART == 2)
          sh.st[1][rt * kTile + row_of(i, hh)][col] = from_f32<T>(sacc[rt][i] - to_f32(hi));
      }
    float vk[FM::PPW][16], vq[FM::PPW][16];
    FM::logits(wop, kop, w, li, hh, vk, sh.fk);
    FM::logits(wop, qop, w, li, hh, vq, sh.fq);

    // In-block softmax branch (keys in rows, queries in columns).
    f32x16 acc_sm = {};
    float m, den;
    {
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
    FM::exps(w, li, hh, vq, sh.fq);
    lds_barrier();
    FM::scale(w, li, vk, sh.fk);
    FM::scale(w, li, vq, sh.fq);
    {
      float lz = 0.0f;
#pragma unroll
      for (int j = 0; j < RPW; ++j) {
        const int p = w + j * NW;
        if (p >= NRT) continue;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = p * kTile + row_of(i, hh);
          const float xk = row_ok ? vk[j][i] : 0.0f;
          const T hi = from_f32<T>(xk);
          sh.phiKT[0][r][li] = hi;
          if constexpr (C::NPART == 2) sh.phiKT[1][r][li] = from_f32<T>(xk - to_f32(hi));
          const T qh = from_f32<T>(vq[j][i]);
          sh.phiQ[0][li][r] = qh;
          if constexpr (C::NPART == 2) sh.phiQ[1][li][r] = from_f32<T>(vq[j][i] - to_f32(qh));
          lz += vq[j][i] * sh.z[r];
        }
      }
      lz += xor32(lz);
      if (hh == 0) sh.lden[w][li] = lz;
    }
    lds_barrier();

    // Readout against the state of the blocks before this one.
    f32x16 acc_lin = {};
    float lden = 0.0f;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) lden += sh.lden[ww][li];
    // (both operands as hi + lo pairs on the bf16 path: hi*hi + lo*hi + hi*lo)
#pragma unroll
    for (int ks = 0; ks < f / KW; ++ks) {
      const op_t pb = lds_op_perm<T>(&sh.phiQ[0][li][0], ks, hh, 0);
      const int rt = ks / C::KL, kk = ks % C::KL;
      acc_lin = M::mma(acc_op<T>(sacc[rt], kk), pb, acc_lin);
      if constexpr (C::NPART == 2) {
        acc_lin = M::mma(acc_op_lo<T>(sacc[rt], kk), pb, acc_lin);
        acc_lin = M::mma(acc_op<T>(sacc[rt], kk), lds_op_perm<T>(&sh.phiQ[1][li][0], ks, hh, 0),
                         acc_lin);
      }
    }
    // Merge (scaled by exp(-c) so nothing overflows): out = N / D with
    // w sm_den = exp(la) den, lin_den = exp(lb), c = max(la, lb).
    float ca = 1.0f, cz = 0.0f, rz = 0.0f, cmax = lw + m;
    if (lden > 0.0f) {
      const float la = lw + m, lb = logf(lden);
      cmax = fmaxf(la, lb);
      ca = expf(la - cmax);
      cz = expf(lb - cmax);
      rz = 1.0f / lden;
    }
    const float inv = 1.0f / (ca * den + cz);
    // upstream gradient (or the teacher's output): query li, columns
    // 32w + row_of(i, hh)
    float gq[16];
    float go_p = 0.0f, gs_p = 0.0f;
    const T* gsrc = (const T*)(tmode ? a.target : a.dout) +
                    (((size_t)b * T_ + t0 + lrow) * Hq + h) * D + w * kTile;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float gin = row_ok ? to_f32(gsrc[row_of(i, hh)]) : 0.0f;
      const float o = (ca * acc_sm[i] + cz * (acc_lin[i] * rz)) * inv;
      if (tmode) {
        const float e = row_ok ? o - gin : 0.0f;
        lss += e * e;
        gq[i] = 2.0f * e;
      } else {
        gq[i] = gin;
      }
      go_p += gq[i] * o;
      gs_p += gq[i] * acc_sm[i];
    }
    go_p += xor32(go_p);
    gs_p += xor32(gs_p);
    if (hh == 0) {
      sh.red[w][li][0] = go_p;
      sh.red[w][li][1] = gs_p;
    }
    lds_barrier();
    float go = 0.0f, gs = 0.0f;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) {
      go += sh.red[ww][li][0];
      gs += sh.red[ww][li][1];
    }
    // 1/D = inv exp(-c); dL/dalpha = dL/dw w(1-w), and
    // dL/dw = exp(m - c) inv (g.acc_sm - (g.out) den) with exp(m - c) w = ca.
    const float rD = inv * expf(-cmax);
    const float gD = -rD * go;
    if (w == 0 && hh == 0 && row_ok) dal += ca * one_minus_w * inv * (gs - go * den);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float x = rD * gq[i];
      const T hi = from_f32<T>(x);
      sh.gn[0][li][w * kTile + row_of(i, hh)] = hi;
      if constexpr (C::NPART == 2) sh.gn[1][li][w * kTile + row_of(i, hh)] = from_f32<T>(x - to_f32(hi));
    }
    if (w == 0 && hh == 0) sh.gd[li] = row_ok ? gD : 0.0f;
    lds_barrier();

    // dL/dN^T and dL/dD for the reverse pass: 8 queries of one column per
    // item, written contiguously.
    {
      float* gnT = ka.gnT + ((size_t)u * ka.nblk + blk) * D * kTile;
      for (int it = tid; it < D * 4; it += blockDim.x) {
        const int c = it >> 2, i0 = (it & 3) * 8;
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          x[e] = to_f32(sh.gn[0][i0 + e][c]);
          if constexpr (C::NPART == 2) x[e] += to_f32(sh.gn[1][i0 + e][c]);
        }
        f32x4* dst = reinterpret_cast<f32x4*>(gnT + (size_t)c * kTile + i0);
        dst[0] = f32x4{x[0], x[1], x[2], x[3]};
        dst[1] = f32x4{x[4], x[5], x[6], x[7]};
      }
      if (tid < kTile) ka.gd[((size_t)u * ka.nblk + blk) * kTile + tid] = sh.gd[tid];
    }

    // dL/dphi(q_i) for the feature tiles this wave owns: rows r of tile p,
    // columns i; S_{c-1} rows from LDS are the A operand (contraction over d).
    float dphi[RPW][16];
#pragma unroll
    for (int j = 0; j < RPW; ++j) {
      const int p = w + j * NW;
      if (p >= NRT) continue;
      f32x16 dq = {};
#pragma unroll
      for (int s = 0; s < NW; ++s)
#pragma unroll
        for (int ks = 0; ks < C::KL; ++ks)
        {
          const op_t ah = lds_op_perm<T>(&sh.st[0][p * kTile + li][0], ks, hh, s * kTile);
          const op_t bh = lds_op_perm<T>(&sh.gn[0][li][0], ks, hh, s * kTile);
          dq = M::mma(ah, bh, dq);
          if constexpr (C::NPART == 2) {
            dq = M::mma(lds_op_perm<T>(&sh.st[1][p * kTile + li][0], ks, hh, s * kTile), bh, dq);
            dq = M::mma(ah, lds_op_perm<T>(&sh.gn[1][li][0], ks, hh, s * kTile), dq);
          }
        }
      const float gdi = sh.gd[li];
      float js = 0.0f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        dphi[j][i] = dq[i] + gdi * sh.z[p * kTile + row_of(i, hh)];
        js += dphi[j][i] * vq[j][i];
      }
      js += xor32(js);
      if (hh == 0) sh.jsum[p][li] = js;
    }
    lds_barrier();
    // Feature-map backward: dL/du for each sign, transposed into LDS.
#pragma unroll
    for (int j = 0; j < RPW; ++j) {
      const int p = w + j * NW;
      if (p >= NRT) continue;
      const int sg = p / NT, t = p % NT;
      float ssum = 0.0f;
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) ssum += sh.jsum[sg * NT + tt][li];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float du = row_ok ? vq[j][i] * (dphi[j][i] - ssum) : 0.0f;
        if (sg) du = -du;
        const int jr = t * kTile + row_of(i, hh);
        const T hi = from_f32<T>(du);
        sh.duT[sg][0][jr][li] = hi;
        if constexpr (C::NPART == 2) sh.duT[sg][1][jr][li] = from_f32<T>(du - to_f32(hi));
      }
    }
    op_t qtop[C::KL];
#pragma unroll
    for (int ks = 0; ks < C::KL; ++ks)
      qtop[ks] = load_rows_op<T>(qb + col, qstride, ks, hh, L, false);
    lds_barrier();
    if constexpr (IN) {
      // dL/du of the block's queries, both signs summed, for dL/dq = W dL/du
      float* dst = ka.duq + ((size_t)u * T_ + t0) * F;
      for (int it = tid; it < L * (F / 4); it += blockDim.x) {
        const int t = it / (F / 4), j4 = (it % (F / 4)) * 4;
        f32x4 x;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float acc = 0.0f;
#pragma unroll
          for (int sg = 0; sg < 2; ++sg)
#pragma unroll
            for (int part = 0; part < C::NPART; ++part) acc += to_f32(sh.duT[sg][part][j4 + e][t]);
          x[e] = acc;
        }
        *reinterpret_cast<f32x4*>(dst + (size_t)t * F + j4) = x;
      }
    }
    // dW^T tiles (rows j of tile t, columns 32w..): += dL/du^T Q.
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int sg = 0; sg < 2; ++sg)
#pragma unroll
        for (int part = 0; part < C::NPART; ++part)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks)
            dwacc[t] = M::mma(lds_op_perm<T>(&sh.duT[sg][part][t * kTile + li][0], ks, hh, 0),
                              qtop[ks], dwacc[t]);
    // Commit the block into S (columns 32w..).
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
      for (int ks = 0; ks < C::KL; ++ks)
#pragma unroll
        for (int part = 0; part < C::NPART; ++part)
          sacc[rt] = M::mma(lds_op_perm<T>(&sh.phiKT[part][rt * kTile + li][0], ks, hh, 0),
                            vop[ks], sacc[rt]);
    // z += sum_t phi(k_t) (every reader of z in this block is past the last
    // barrier).
    for (int r = tid; r < f; r += blockDim.x) {
      float s = 0.0f;
#pragma unroll
      for (int part = 0; part < C::NPART; ++part)
        for (int t = 0; t < kTile; ++t) s += to_f32(sh.phiKT[part][r][t]);
      sh.z[r] += s;
    }
  }

  // Partials of this (request, head, segment).
  float* dwq = ka.dwq + ((size_t)u * nseg + seg) * F * D;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int i = 0; i < 16; ++i) dwq[(size_t)(t * kTile + row_of(i, hh)) * D + col] = dwacc[t][i];
  dal = wave_sum(dal);
  lss = wave_sum(lss);
  if (lane == 0) {
    sh.fin[w][0] = dal;
    sh.fin[w][1] = lss;
  }
  lds_barrier();
  if (tid == 0) {
    float x0 = 0.0f, x1 = 0.0f;
    for (int ww = 0; ww < NW; ++ww) {
      x0 += sh.fin[ww][0];
      x1 += sh.fin[ww][1];
    }
    ka.red[((size_t)u * nseg + seg) * 2] = x0;
    ka.red[((size_t)u * nseg + seg) * 2 + 1] = x1;
  }
}


// ---------------------------------------------------------------------------
// 2'. Pipelined forward walk (bf16, F <= 64).  Producers prepare block c+1
// while the state waves finish block c:
//   wave 0: phi(Q) as packed hi/lo pairs [query][feature] (the readout's
//           operand, and phi(Q) itself for the feature-map Jacobian), and
//           lin_den = phi(Q) z in fp32 from the map's registers;
//   wave 1: phi(K) transposed and packed (the commit's operand), and
//           z_{c+1} = z_c + sum_t phi(k_t) from its previous map;
//   waves 2 .. NP-1: the in-block softmax numerators P V (relative to the
//           row maximum) for 64 columns each, the row maxima and sums, and
//           the V^T operands of the commit; then, once the state waves have
//           posted dL/du of their block, the query part of dW for the same
//           64 columns;
//   state waves (D/32): S columns 32w..32w+31 (the readout) and S^T for the
//           feature tiles w, w + D/32, ... (dL/dphi(Q), which contracts over
//           the head dimension) both in fp32 accumulators; the merge, dL/dN,
//           dL/dD, dL/dphi(Q) and dL/du; then the commit of the block into
//           both copies.
// Four barriers per block, all waves: after the merge's partial sums, after
// dL/dN, after the per-sign sums and after dL/du.  The producers do their
// block's work after the first barrier (the z update aside), which also
// makes an end-of-step barrier unnecessary: the buffer that the state waves'
// commit reads is refilled only after the next first barrier, and the
// softmax waves' dW, which reads dL/du, ends before they reach it.
// ---------------------------------------------------------------------------
template <int D, int F>
struct FPipeCfg {
  typedef Mma<bf16> M;
  typedef typename M::op_t op_t;
  static constexpr int NC = D / kTile;                 // state waves
  static constexpr int NSM = D / 64 > 0 ? D / 64 : 1;  // softmax waves
  static constexpr int CT = NC / NSM;                  // column tiles per softmax wave
  static constexpr int NP = 2 + NSM;
  static constexpr int NWAVE = NP + NC;
  static constexpr int f = 2 * F;
  static constexpr int NRT = f / kTile;
  static constexpr int NT = F / kTile;
  static constexpr int RPW = (NRT + NC - 1) / NC;      // S^T feature tiles per state wave
  static constexpr int KD = D / M::KW;
  static constexpr int KL = kTile / M::KW;
  static constexpr int KF = f / M::KW;
  typedef WaveFeatMap<bf16, D, F> WFM;
  struct alignas(16) Buf {
    uint32_t phiQ[kTile][f + 4];     // phi(q_i)[r] at [i][r], bf16 hi | lo << 16
    uint32_t phiKT[f][kTile + 4];    // phi(k_t)[r] at [r][t], packed likewise
    float sm[kTile][D + 4];          // P V relative to the row maximum, [i][c]
    float m[kTile], den[kTile];
    op_t vop[NC][KL][kWave];         // V^T: lane (c, hh), tokens in row_of order
    op_t qtop[NC][KL][kWave];        // Q^T likewise
  };
  struct alignas(16) Smem {
    Buf buf[2];
    union {
      uint32_t gn[kTile][D + 4];     // dL/dN_i[c] at [i][c], packed
      uint32_t duT[2][F][kTile + 4]; // +-dL/du of each sign at [j][t], packed
    } x;
    float z[2][f];                   // z before block blk0 + n at [n & 1]
    float lden[2][kTile];            // phi(q_i) . z of block blk0 + n at [n & 1]
    float red[NC][kTile][2];
    float jsum[NRT][kTile];
    float fin[NC][2];
  };
};

template <int D>
constexpr int fpipe_threads() {
  return kWave * (2 + (D / 64 > 0 ? D / 64 : 1) + D / kTile);
}

template <int D, int F>
__global__ __launch_bounds__(fpipe_threads<D>()) void hyb_bwd_fpipe_kernel(BwdKArgs ka) {
  typedef FPipeCfg<D, F> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  typedef typename C::WFM WFM;
  typedef typename C::Buf Buf;
  constexpr int f = C::f, E = M::E, KW = M::KW, NP = C::NP, NC = C::NC;
  constexpr int NRT = C::NRT, NT = C::NT, RPW = C::RPW, KD = C::KD, KL = C::KL;
  constexpr int NBAR = 4;  // barriers per block step
  static_assert(fpipe_threads<D>() == kWave * C::NWAVE, "launch bounds match the waves");
  __shared__ typename C::Smem sh;
  const BackwardArgs& a = ka.a;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L, T_ = a.T;
  const int units = a.s.B * Hq, nseg = ka.nseg;
  const int vix = xcd_unit(blockIdx.x, units * nseg);
  const int u = vix % units, seg = vix / units;
  const int b = u / Hq, h = u % Hq, g = h / (Hq / Hkv);
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
  const int blk0 = seg * ka.seg_blocks, blk1 = min(ka.nblk, blk0 + ka.seg_blocks);
  const int nb = blk1 - blk0;
  const bool row_ok = li < L;
  const int lrow = min(li, L - 1);
  auto qbase = [&](int blk) {
    return (const bf16*)a.q + (((size_t)b * T_ + (size_t)blk * L) * Hq + h) * D;
  };
  auto kbase = [&](int blk) {
    return (const bf16*)a.k + (((size_t)b * T_ + (size_t)blk * L) * Hkv + g) * D;
  };
  auto vbase = [&](int blk) {
    return (const bf16*)a.v + (((size_t)b * T_ + (size_t)blk * L) * Hkv + g) * D;
  };
  auto load_rows = [&](const bf16* base, size_t stride, op_t (&o)[KD]) {
    const bf16* row = base + (size_t)lrow * stride + hh * E;
#pragma unroll
    for (int ks = 0; ks < KD; ++ks) o[ks] = load_op<bf16>(row + ks * KW);
  };

  // z at the segment's start: the earlier segments' sums
  for (int r = tid; r < f; r += blockDim.x) {
    float zr = 0.0f;
    for (int pc = 0; pc < seg * ka.ppseg; ++pc) zr += ka.dz[((size_t)u * ka.npc + pc) * f + r];
    sh.z[0][r] = zr;
  }
  // dL/du and the second buffer's Q^T operands start at zero: the softmax
  // waves' first dW update then adds exact zeros, and their loop needs no
  // branch (which would make the compiler keep a second copy of dW)
  for (int i = tid; i < (int)(sizeof(sh.x) / 4); i += blockDim.x) reinterpret_cast<uint32_t*>(&sh.x)[i] = 0u;
  for (int i = tid; i < (int)(sizeof(sh.buf[1].qtop) / 4); i += blockDim.x)
    reinterpret_cast<uint32_t*>(&sh.buf[1].qtop)[i] = 0u;
  lds_barrier();

  if (w < 2) {
    // ---- feature map of Q (wave 0) or K (wave 1) ----
    const bf16* __restrict__ Wt_h = (const bf16*)a.W + (size_t)h * F * D;
    op_t wop[WFM::NT][KD];
    WFM::load_w(Wt_h, li, hh, wop);
    op_t x[KD];
    auto load = [&](int blk) {
      if (w == 0) load_rows(qbase(blk), qstride, x);
      else load_rows(kbase(blk), kstride, x);
    };
    if (nb > 0) load(blk0);
    // Block blk0 + n is prepared in iteration n, after the state waves'
    // first barrier: their readout and merge phase, the longest of the step
    // and the one with the most VALU work, then has the SIMDs it shares with
    // this wave to itself.  Only the K wave's z update runs before it.
    for (int n = 0; n <= nb; ++n) {
      if (w == 1 && n > 0 && n < nb) {
        // z before block blk0 + n: z before the previous block plus the sum
        // of its phi(k_t), from the map this wave stored an iteration ago (a
        // padding key's phi is stored as zero)
        const Buf& Bp = sh.buf[(n - 1) & 1];
        const float* zp = sh.z[(n - 1) & 1];
        float* zn = sh.z[n & 1];
#pragma unroll
        for (int r = lane; r < f; r += kWave) {
          float zs = zp[r];
#pragma unroll
          for (int t0 = 0; t0 < kTile; t0 += 4) {
            const uint4 xk = *reinterpret_cast<const uint4*>(&Bp.phiKT[r][t0]);
#pragma unroll
            for (int e = 0; e < 4; ++e) zs += unpack_hi(xk[e]) + unpack_lo(xk[e]);
          }
          zn[r] = zs;
        }
      }
      lds_barrier();  // 1
      // (phi stays in registers past the second barrier: wave 0 forms
      // lin_den from it there)
      float phi[WFM::NPAIR][16];
      if (n < nb) {
        Buf& B = sh.buf[n & 1];
        // a padding row reads row L-1 (finite); keep = row_ok zeroes its phi
        WFM::logits(wop, x, phi);
        if (n + 1 < nb) load(blk0 + n + 1);
        WFM::softmax(phi, row_ok);
        if (w == 0) {
#pragma unroll
          for (int p = 0; p < WFM::NPAIR; ++p)
#pragma unroll
            for (int i = 0; i < 16; i += 4) {
              uint4 pk;
              pack_hi_lo2(phi[p][i], phi[p][i + 1], pk[0], pk[1]);
              pack_hi_lo2(phi[p][i + 2], phi[p][i + 3], pk[2], pk[3]);
              *reinterpret_cast<uint4*>(&B.phiQ[li][WFM::feature(16 * p + i, hh)]) = pk;
            }
        } else {
#pragma unroll
          for (int p = 0; p < WFM::NPAIR; ++p)
#pragma unroll
            for (int i = 0; i < 16; i += 2)
              pack_hi_lo2(phi[p][i], phi[p][i + 1], B.phiKT[WFM::feature(16 * p + i, hh)][li],
                          B.phiKT[WFM::feature(16 * p + i + 1, hh)][li]);
        }
      }
      lds_barrier();  // 2
      if (w == 0 && n < nb) {
        // lin_den = phi(q_li) . z of block blk0 + n, in fp32 from the map's
        // registers, for the state waves' merge an iteration later (z was
        // posted by the K wave before the first barrier)
        const float* zn = sh.z[n & 1];
        float part = 0.0f;
#pragma unroll
        for (int p = 0; p < WFM::NPAIR; ++p)
#pragma unroll
          for (int i = 0; i < 16; i += 4) {
            const f32x4 z4 = *reinterpret_cast<const f32x4*>(&zn[WFM::feature(16 * p + i, hh)]);
#pragma unroll
            for (int e = 0; e < 4; ++e) part += phi[p][i + e] * z4[e];
          }
        part += xor32(part);
        if (hh == 0) sh.lden[n & 1][li] = part;
      }
#pragma unroll
      for (int k = 2; k < NBAR; ++k) lds_barrier();
    }
  } else if (w < NP) {
    // ---- in-block softmax branch for column tiles c0 .. c0+CT-1 ----
    const int c0 = (w - 2) * C::CT;
    const float scale = 1.0f / sqrtf((float)D);
    // K, Q and V rows through buffer descriptors over the request's rows (a
    // scalar base, a 32-bit lane offset, the block as a scalar offset; the
    // launcher keeps them under 2 GiB): 64-bit lane addresses kept across
    // the step would spill, and each reload from scratch would wait for the
    // next block's loads in flight.  V comes as rows too, 16 bytes of this
    // wave's columns per lane and k-step, and is turned into V^T operands by
    // the identity product, like Q^T.
    const __amdgpu_buffer_rsrc_t qrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>((const bf16*)a.q + (size_t)b * T_ * qstride), 0,
        (int)(T_ * qstride * sizeof(bf16)), kBufferWord3);
    const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>((const bf16*)a.k + (size_t)b * T_ * kstride), 0,
        (int)(T_ * kstride * sizeof(bf16)), kBufferWord3);
    const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>((const bf16*)a.v + (size_t)b * T_ * kstride), 0,
        (int)(T_ * kstride * sizeof(bf16)), kBufferWord3);
    const int qlane = (int)(((size_t)lrow * qstride + (size_t)h * D + hh * E) * sizeof(bf16));
    const int klane = (int)(((size_t)lrow * kstride + (size_t)g * D + hh * E) * sizeof(bf16));
    op_t ko[KD], qo[KD], vr[C::CT][KL];
    auto load = [&](int blk) {
      const int qso = (int)((size_t)blk * L * qstride * sizeof(bf16));
      const int kso = (int)((size_t)blk * L * kstride * sizeof(bf16));
#pragma unroll
      for (int ks = 0; ks < KD; ++ks) ko[ks] = buf_op<bf16>(krs, klane + ks * KW * (int)sizeof(bf16), kso);
#pragma unroll
      for (int ks = 0; ks < KD; ++ks) qo[ks] = buf_op<bf16>(qrs, qlane + ks * KW * (int)sizeof(bf16), qso);
#pragma unroll
      for (int ct = 0; ct < C::CT; ++ct)
#pragma unroll
        for (int kk = 0; kk < KL; ++kk)
          vr[ct][kk] = buf_op<bf16>(vrs, klane + ((c0 + ct) * kTile + kk * KW) * (int)sizeof(bf16), kso);
    };
    // the identity's k-steps: B[k][n] = (k == n) for n = li
    op_t idop[KL];
#pragma unroll
    for (int kk = 0; kk < KL; ++kk)
#pragma unroll
      for (int e = 0; e < E; ++e) idop[kk][e] = (bf16)(kk * KW + hh * E + e == li ? 1.0f : 0.0f);
    // the query part of dW^T for columns 32(c0+ct)..: rows j of tile t
    f32x16 dwacc[NT][C::CT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int ct = 0; ct < C::CT; ++ct) dwacc[t][ct] = f32x16{};
    if (nb > 0) load(blk0);
    for (int n = 0; n <= nb; ++n) {
      // block blk0 + n after the state waves' first barrier, as for the
      // feature maps
      lds_barrier();  // 1
      if (n < nb) {
        Buf& B = sh.buf[n & 1];
        // keys in rows, queries in columns
        f32x16 sc = {};
#pragma unroll
        for (int ks = 0; ks < KD; ++ks)
          sc = M::mma(keep_if<bf16>(row_ok, ko[ks]), keep_if<bf16>(row_ok, qo[ks]), sc);
        // Q^T operands (lane: column, elements: tokens in row_of order) from
        // the Q rows times the identity: Q_c = Q_c I holds the tokens in its
        // accumulator rows (exact: one nonzero bf16 product per entry)
        // (this wave's column tiles picked with constant indices: the wave
        // index is uniform but not a compile-time constant)
        op_t qsel[C::CT][KL];
#pragma unroll
        for (int sw = 0; sw < C::NSM; ++sw)
          if (w - 2 == sw) {
#pragma unroll
            for (int ct = 0; ct < C::CT; ++ct)
#pragma unroll
              for (int kk = 0; kk < KL; ++kk) qsel[ct][kk] = qo[(sw * C::CT + ct) * KL + kk];
          }
        op_t vo[C::CT][KL];
#pragma unroll
        for (int ct = 0; ct < C::CT; ++ct) {
          f32x16 qa = {}, va = {};
#pragma unroll
          for (int kk = 0; kk < KL; ++kk) {
            qa = M::mma(keep_if<bf16>(row_ok, qsel[ct][kk]), idop[kk], qa);
            va = M::mma(keep_if<bf16>(row_ok, vr[ct][kk]), idop[kk], va);
          }
#pragma unroll
          for (int kk = 0; kk < KL; ++kk) {
            B.qtop[c0 + ct][kk][lane] = acc_op<bf16>(qa, kk);
            vo[ct][kk] = acc_op<bf16>(va, kk);
          }
        }
        float pr[16];
        float m = -INFINITY;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          pr[i] = row_of(i, hh) < L ? sc[i] * scale : -INFINITY;
          m = fmaxf(m, pr[i]);
        }
        m = fmaxf(m, xor32(m));
        float den = 0.0f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          pr[i] = row_of(i, hh) < L ? fast_exp(pr[i] - m) : 0.0f;
          den += pr[i];
        }
        den += xor32(den);
#pragma unroll
        for (int ct = 0; ct < C::CT; ++ct) {
          f32x16 acc = {};
#pragma unroll
          for (int ks = 0; ks < KL; ++ks) acc = mma_split_b<bf16>(vo[ct][ks], &pr[ks * E], acc);
#pragma unroll
          for (int i = 0; i < 16; i += 4)
            *reinterpret_cast<f32x4*>(&B.sm[li][(c0 + ct) * kTile + row_of(i, hh)]) =
                f32x4{acc[i], acc[i + 1], acc[i + 2], acc[i + 3]};
        }
        if (w == 2 && hh == 0) {
          B.m[li] = m;
          B.den[li] = den;
        }
#pragma unroll
        for (int ct = 0; ct < C::CT; ++ct)
#pragma unroll
          for (int ks = 0; ks < KL; ++ks) B.vop[c0 + ct][ks][lane] = vo[ct][ks];
        if (n + 1 < nb) load(blk0 + n + 1);  // next block in flight
      }
#pragma unroll
      for (int k = 1; k < NBAR; ++k) lds_barrier();
      {
        // dW^T += dL/du^T Q for the block the state waves are finishing
        // (its dL/du is in LDS from their fourth barrier until they post the
        // next block's dL/dN after the next first barrier; zeros at n = 0)
        const Buf& Bp = sh.buf[(n - 1) & 1];
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int sg = 0; sg < 2; ++sg)
#pragma unroll
            for (int ks = 0; ks < KL; ++ks) {
              op_t uh, ul;
              lds_pair_op(&sh.x.duT[sg][t * kTile + li][0], ks, hh, uh, ul);
#pragma unroll
              for (int ct = 0; ct < C::CT; ++ct) {
                const op_t qt = Bp.qtop[c0 + ct][ks][lane];
                dwacc[t][ct] = M::mma(uh, qt, dwacc[t][ct]);
                dwacc[t][ct] = M::mma(ul, qt, dwacc[t][ct]);
              }
            }
        if (ka.duq != nullptr && n > 0) {
          // with the input gradients: dL/du of the same block's queries, both
          // signs summed (each as its pair hi + lo), for dL/dq = W_h dL/du
          float* dst = ka.duq + ((size_t)u * T_ + (size_t)(blk0 + n - 1) * L) * F;
          for (int it = (w - 2) * kWave + lane; it < L * (F / 4); it += C::NSM * kWave) {
            const int t = it / (F / 4), j4 = (it % (F / 4)) * 4;
            f32x4 x;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float acc = 0.0f;
#pragma unroll
              for (int sg = 0; sg < 2; ++sg) {
                const uint32_t pk = sh.x.duT[sg][j4 + e][t];
                acc += unpack_hi(pk);
                acc += unpack_lo(pk);
              }
              x[e] = acc;
            }
            *reinterpret_cast<f32x4*>(dst + (size_t)t * F + j4) = x;
          }
        }
      }
    }
    float* dwq = ka.dwq + ((size_t)u * nseg + seg) * F * D;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int ct = 0; ct < C::CT; ++ct)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          dwq[(size_t)(t * kTile + row_of(i, hh)) * D + (c0 + ct) * kTile + li] = dwacc[t][ct][i];
  } else {
    // ---- state waves ----
    const int cw = w - NP, col = cw * kTile + li;
    const bool tmode = a.target != nullptr;
    const float lw = log_sigmoid(a.alpha[h]);
    const float one_minus_w = expf(log_sigmoid(-a.alpha[h]));
    // S (columns col) and S^T (feature tiles cw + j*NC): the earlier
    // segments' increments
    // (the first increment is loaded straight into the accumulators, so all
    // its loads are in flight at once; the others are added one by one)
    f32x16 sacc[NRT], sT[RPW][NC];
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) sacc[rt] = f32x16{};
#pragma unroll
    for (int j = 0; j < RPW; ++j)
#pragma unroll
      for (int s = 0; s < NC; ++s) sT[j][s] = f32x16{};
    auto add_increment = [&](int pc, bool first) {
      const float* src = ka.dS + ((size_t)u * ka.npc + pc) * D * f;
#pragma unroll
      for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
        for (int i = 0; i < 16; i += 4) {
          const f32x4 y = *reinterpret_cast<const f32x4*>(src + (size_t)col * f + rt * kTile + row_of(i, hh));
#pragma unroll
          for (int e = 0; e < 4; ++e) sacc[rt][i + e] = first ? y[e] : sacc[rt][i + e] + y[e];
        }
#pragma unroll
      for (int j = 0; j < RPW; ++j) {
        const int p = cw + j * NC;
        if (p >= NRT) continue;
#pragma unroll
        for (int s = 0; s < NC; ++s)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const float y = src[(size_t)(s * kTile + row_of(i, hh)) * f + p * kTile + li];
            sT[j][s][i] = first ? y : sT[j][s][i] + y;
          }
      }
    };
    if (seg > 0) add_increment(0, true);
    for (int pc = 1; pc < seg * ka.ppseg; ++pc) add_increment(pc, false);
    float dal = 0.0f, lss = 0.0f;
    // the block's upstream rows (dout, or the teacher's output) at columns
    // 32cw + row_of(i, hh): prefetched a block ahead
    // Global accesses of this role go through buffer descriptors (a scalar
    // base per request or unit, a 32-bit lane offset, the block as a scalar
    // offset; the launcher keeps each range under 2 GiB): 64-bit lane
    // addresses kept across the step would spill, and every reload from
    // scratch waits for all outstanding memory operations.
    const __amdgpu_buffer_rsrc_t grs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>((const bf16*)(tmode ? a.target : a.dout) + (size_t)b * T_ * qstride), 0,
        (int)(T_ * qstride * sizeof(bf16)), kBufferWord3);
    const int glane = (int)(((size_t)lrow * qstride + (size_t)h * D + cw * kTile + 4 * hh) * sizeof(bf16));
    const __amdgpu_buffer_rsrc_t nrs = __builtin_amdgcn_make_buffer_rsrc(
        ka.gnT + (size_t)u * ka.nblk * D * kTile, 0, (int)((size_t)ka.nblk * D * kTile * sizeof(float)),
        kBufferWord3);
    const int nlane = (int)(((cw * kTile + 4 * hh) * kTile + li) * sizeof(float));
    const __amdgpu_buffer_rsrc_t drs = __builtin_amdgcn_make_buffer_rsrc(
        ka.gd + (size_t)u * ka.nblk * kTile, 0, (int)((size_t)ka.nblk * kTile * sizeof(float)), kBufferWord3);
    bf16x4 gin4[4];
    auto load_g = [&](int blk) {
      const int so = (int)((size_t)blk * L * qstride * sizeof(bf16));
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4)
        gin4[i4] = __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(grs, glane + 16 * i4, so, 0));
    };
    if (nb > 0) load_g(blk0);
    // step 0: the producers fill the first buffer
#pragma unroll
    for (int k = 0; k < NBAR; ++k) lds_barrier();
    for (int n = 1; n <= nb; ++n) {
      const int blk = blk0 + n - 1;
      Buf& B = sh.buf[(n - 1) & 1];
      const int zb = (n - 1) & 1;
      const float* zc = sh.z[zb];
      // -- readout against S_{c-1}, both operands as hi + lo pairs;
      // lin_den = phi(q) . z_{c-1} from the phi(Q) wave
      f32x16 acc_lin = {};
#pragma unroll
      for (int ks = 0; ks < C::KF; ++ks) {
        op_t ph, pl;
        lds_pair_op(&B.phiQ[li][0], ks, hh, ph, pl);
        const int rt = ks / KL, kk = ks % KL;
        op_t sa, sl;
        acc_op_pair(sacc[rt], kk, sa, sl);
        acc_lin = M::mma(sa, ph, acc_lin);
        acc_lin = M::mma(sl, ph, acc_lin);
        acc_lin = M::mma(sa, pl, acc_lin);
      }
      const float lden = sh.lden[zb][li];
      // -- merge (scaled by exp(-c) so nothing overflows): out = N / D with
      // w sm_den = exp(la) den, lin_den = exp(lb), c = max(la, lb)
      const float m = B.m[li], den = B.den[li];
      float ca = 1.0f, cz = 0.0f, rz = 0.0f, cmax = lw + m;
      if (lden > 0.0f) {
        const float la = lw + m, lb = logf(lden);
        cmax = fmaxf(la, lb);
        ca = expf(la - cmax);
        cz = expf(lb - cmax);
        rz = 1.0f / lden;
      }
      const float inv = 1.0f / (ca * den + cz);
      float gq[16];
      float go_p = 0.0f, gs_p = 0.0f;
#pragma unroll
      for (int i4 = 0; i4 < 16; i4 += 4) {
        const f32x4 smv = *reinterpret_cast<const f32x4*>(&B.sm[li][col - li + row_of(i4, hh)]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = i4 + e;
          const float gin = row_ok ? (float)gin4[i4 / 4][e] : 0.0f;
          const float o = (ca * smv[e] + cz * (acc_lin[i] * rz)) * inv;
          if (tmode) {
            const float er = row_ok ? o - gin : 0.0f;
            lss += er * er;
            gq[i] = 2.0f * er;
          } else {
            gq[i] = gin;
          }
          go_p += gq[i] * o;
          gs_p += gq[i] * smv[e];
        }
      }
      if (n < nb) load_g(blk + 1);
      go_p += xor32(go_p);
      gs_p += xor32(gs_p);
      if (hh == 0) {
        sh.red[cw][li][0] = go_p;
        sh.red[cw][li][1] = gs_p;
      }
      lds_barrier();  // 1
      // -- dL/dN (packed, and fp32 for the reverse pass), dL/dD, dL/dalpha
      float go = 0.0f, gs = 0.0f;
#pragma unroll
      for (int ww = 0; ww < NC; ++ww) {
        go += sh.red[ww][li][0];
        gs += sh.red[ww][li][1];
      }
      // 1/D = inv exp(-c); dL/dalpha = dL/dw w(1-w), and
      // dL/dw = exp(m - c) inv (g.acc_sm - (g.out) den) with exp(m - c) w = ca.
      const float rD = inv * expf(-cmax);
      const float gD = row_ok ? -rD * go : 0.0f;
      if (cw == 0 && hh == 0 && row_ok) dal += ca * one_minus_w * inv * (gs - go * den);
      {
        // dL/dN^T: column 32cw + row_of(i, hh) = 32cw + 4hh + 8(i/4) + i%4,
        // query li; the lane's offset, the block's, the rest immediate
        const int nso = (int)((size_t)blk * D * kTile * sizeof(float));
#pragma unroll
        for (int i4 = 0; i4 < 16; i4 += 4) {
          uint4 pk;
          float x[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            x[e] = rD * gq[i4 + e];
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, x[e]), nrs,
                                                  nlane + (2 * i4 + e) * kTile * (int)sizeof(float), nso, 0);
          }
          pack_hi_lo2(x[0], x[1], pk[0], pk[1]);
          pack_hi_lo2(x[2], x[3], pk[2], pk[3]);
          *reinterpret_cast<uint4*>(&sh.x.gn[li][col - li + row_of(i4, hh)]) = pk;
        }
        if (cw == 0 && hh == 0)
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, gD), drs, li * (int)sizeof(float),
                                                (int)(blk * kTile * sizeof(float)), 0);
      }
      lds_barrier();  // 2
      // -- dL/dphi(q_i) = S_{c-1} dL/dN_i + z_{c-1} dL/dD_i for the feature
      // tiles this wave owns (rows r, columns i), and the per-tile sums
      float dphi[RPW][16], pq[RPW][16];
#pragma unroll
      for (int j = 0; j < RPW; ++j) {
        const int p = cw + j * NC;
        if (p >= NRT) continue;
        f32x16 dq = {};
#pragma unroll
        for (int s = 0; s < NC; ++s)
#pragma unroll
          for (int ks = 0; ks < KL; ++ks) {
            op_t gh, gl;
            lds_pair_op(&sh.x.gn[li][s * kTile], ks, hh, gh, gl);
            op_t ah, al;
            acc_op_pair(sT[j][s], ks, ah, al);
            dq = M::mma(ah, gh, dq);
            dq = M::mma(al, gh, dq);
            dq = M::mma(ah, gl, dq);
          }
        float js = 0.0f;
#pragma unroll
        for (int i4 = 0; i4 < 16; i4 += 4) {
          const int r = p * kTile + row_of(i4, hh);
          const uint4 xq = *reinterpret_cast<const uint4*>(&B.phiQ[li][r]);
          const f32x4 z4 = *reinterpret_cast<const f32x4*>(&zc[r]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            pq[j][i4 + e] = unpack_hi(xq[e]) + unpack_lo(xq[e]);
            dphi[j][i4 + e] = dq[i4 + e] + gD * z4[e];
            js += dphi[j][i4 + e] * pq[j][i4 + e];
          }
        }
        js += xor32(js);
        // (the lane index through an opaque copy: an LDS address kept live
        // across the step is spilled, and its reload here would wait for the
        // dL/dN^T stores in flight)
        int lj = li;
        asm volatile("" : "+v"(lj));
        if (hh == 0) sh.jsum[p][lj] = js;
      }
      lds_barrier();  // 3
      // -- feature-map backward: dL/du of each sign, transposed and packed
      // (phi(q) of a padding query is stored as zero, so is its dL/du)
#pragma unroll
      for (int j = 0; j < RPW; ++j) {
        const int p = cw + j * NC;
        if (p >= NRT) continue;
        const int sg = p / NT, t = p % NT;
        float ssum = 0.0f;
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) ssum += sh.jsum[sg * NT + tt][li];
        const float sgn = sg ? -1.0f : 1.0f;
#pragma unroll
        for (int i = 0; i < 16; i += 2)
          pack_hi_lo2(sgn * pq[j][i] * (dphi[j][i] - ssum), sgn * pq[j][i + 1] * (dphi[j][i + 1] - ssum),
                      sh.x.duT[sg][t * kTile + row_of(i, hh)][li],
                      sh.x.duT[sg][t * kTile + row_of(i + 1, hh)][li]);
      }
      lds_barrier();  // 4
      // -- commit the block: S += phi(K)^T V (columns col), S^T += V^T phi(K)
      // (feature tiles of this wave); the K wave forms z_{c+1}
      int lv = lane;  // (an opaque copy, as above)
      asm volatile("" : "+v"(lv));
#pragma unroll
      for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
        for (int ks = 0; ks < KL; ++ks) {
          op_t khi, klo;
          lds_pair_op(&B.phiKT[rt * kTile + li][0], ks, hh, khi, klo);
          const op_t vk = B.vop[cw][ks][lv];
          sacc[rt] = M::mma(khi, vk, sacc[rt]);
          sacc[rt] = M::mma(klo, vk, sacc[rt]);
        }
#pragma unroll
      for (int j = 0; j < RPW; ++j) {
        const int p = cw + j * NC;
        if (p >= NRT) continue;
#pragma unroll
        for (int ks = 0; ks < KL; ++ks) {
          op_t khi, klo;
          lds_pair_op(&B.phiKT[p * kTile + li][0], ks, hh, khi, klo);
#pragma unroll
          for (int s = 0; s < NC; ++s) {
            const op_t vs = B.vop[s][ks][lv];
            sT[j][s] = M::mma(vs, khi, sT[j][s]);
            sT[j][s] = M::mma(vs, klo, sT[j][s]);
          }
        }
      }
    }
    // partials of this (request, head, segment)
    dal = wave_sum(dal);
    lss = wave_sum(lss);
    if (lane == 0) {
      sh.fin[cw][0] = dal;
      sh.fin[cw][1] = lss;
    }
  }
  lds_barrier();
  if (tid == NP * kWave) {
    float x0 = 0.0f, x1 = 0.0f;
    for (int ww = 0; ww < NC; ++ww) {
      x0 += sh.fin[ww][0];
      x1 += sh.fin[ww][1];
    }
    ka.red[((size_t)u * nseg + seg) * 2] = x0;
    ka.red[((size_t)u * nseg + seg) * 2 + 1] = x1;
  }
}

// ---------------------------------------------------------------------------
// 3./4. Reverse walk (delta: only the segment's Gbar sum).
// ---------------------------------------------------------------------------
template <typename T, int D, int F, bool IN>
__global__ __launch_bounds__(kWave*(D / kTile)) void hyb_bwd_rev_kernel(BwdKArgs ka, int delta) {
  typedef BwdCfg<T, D, F> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  typedef typename C::FM FM;
  constexpr int f = C::f, E = M::E, KW = M::KW, NW = C::NW, RPW = C::RPW;
  constexpr int NT = C::NT, NRT = C::NRT;
  __shared__ typename C::SmemB sh;
  __shared__ typename std::conditional<IN, RevInSmem<T, D, F>, NoSmem>::type shi;
  const BackwardArgs& a = ka.a;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);  // wave-uniform
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L, T_ = a.T;
  const int units = a.s.B * Hq, nseg = ka.nseg;
  // delta: one workgroup per (unit, piece of segments 1 .. nseg-1; segment
  // 0's sum is never needed); walk: per (unit, segment)
  const int vix = xcd_unit(blockIdx.x, units * (delta ? ka.npc : nseg));
  const int u = vix % units, seg = vix / units;  // (delta: the piece)
  const int b = u / Hq, h = u % Hq, g = h / (Hq / Hkv);
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
  const int col = w * kTile + li;
  int blk0 = seg * ka.seg_blocks, blk1 = min(ka.nblk, blk0 + ka.seg_blocks);
  if (delta) rev_piece(ka, seg, blk0, blk1);

  // Gbar^T tiles (rows c of slice s, columns of feature tile p) and gz:
  // the sums over the later segments.
  f32x16 gacc[RPW][NW];
#pragma unroll
  for (int j = 0; j < RPW; ++j)
#pragma unroll
    for (int s = 0; s < NW; ++s) gacc[j][s] = f32x16{};
  for (int r = tid; r < f; r += blockDim.x) sh.gz[r] = 0.0f;
  if (!delta) {
    for (int sp = seg * ka.ppseg; sp < ka.npc; ++sp) {
      const float* src = ka.dG + ((size_t)u * ka.npc + sp) * D * f;
#pragma unroll
      for (int j = 0; j < RPW; ++j) {
        const int p = w + j * NW;
        if (p >= NRT) continue;
#pragma unroll
        for (int s = 0; s < NW; ++s)
#pragma unroll
          for (int i = 0; i < 16; ++i)
            gacc[j][s][i] += src[(size_t)(s * kTile + row_of(i, hh)) * f + p * kTile + li];
      }
      const float* zs = ka.dgz + ((size_t)u * ka.npc + sp) * f;
      for (int r = tid; r < f; r += blockDim.x) sh.gz[r] += zs[r];
    }
  }

  const T* __restrict__ Wt_h = (const T*)a.W + (size_t)h * F * D;
  op_t wop[FM::PPW][C::KD];
  FM::load_w(Wt_h, w, li, hh, wop);
  const bool row_ok = li < L;
  const int lrow = min(li, L - 1);
  f32x16 dwacc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) dwacc[t] = f32x16{};

  for (int blk = blk1 - 1; blk >= blk0; --blk) {
    const size_t t0 = (size_t)blk * L;
    const T* kb = (const T*)a.k + (((size_t)b * T_ + t0) * Hkv + g) * D;
    const T* vb = (const T*)a.v + (((size_t)b * T_ + t0) * Hkv + g) * D;
    const T* qb = (const T*)a.q + (((size_t)b * T_ + t0) * Hq + h) * D;
    const float* gnT = ka.gnT + ((size_t)u * ka.nblk + blk) * D * kTile;
    op_t qop[C::KD], kop[C::KD], vrow[NW][C::KL], ktop[C::KL];
    {
      const T* qrow = qb + (size_t)lrow * qstride + hh * E;
#pragma unroll
      for (int ks = 0; ks < C::KD; ++ks) qop[ks] = keep_if<T>(row_ok, load_op<T>(qrow + ks * KW));
      if (!delta) {
        const T* krow = kb + (size_t)lrow * kstride + hh * E;
        const T* vr = vb + (size_t)lrow * kstride;
#pragma unroll
        for (int ks = 0; ks < C::KD; ++ks) kop[ks] = keep_if<T>(row_ok, load_op<T>(krow + ks * KW));
#pragma unroll
        for (int s = 0; s < NW; ++s)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks)
            vrow[s][ks] = keep_if<T>(row_ok, lds_op_perm<T>(vr, ks, hh, s * kTile));
        if constexpr (sizeof(T) == 2) {
          // K^T operands of this wave's columns: its K row operands times
          // the identity (exact), rather than 2-byte gathers (pairs of them
          // share a register, and each waits for the other)
          op_t ksel[C::KL];
#pragma unroll
          for (int sw = 0; sw < NW; ++sw)
            if (w == sw) {
#pragma unroll
              for (int kk = 0; kk < C::KL; ++kk) ksel[kk] = kop[sw * C::KL + kk];
            }
          f32x16 kt = {};
#pragma unroll
          for (int kk = 0; kk < C::KL; ++kk) {
            op_t id;
#pragma unroll
            for (int e = 0; e < E; ++e) id[e] = (T)(kk * KW + hh * E + e == li ? 1.0f : 0.0f);
            kt = M::mma(ksel[kk], id, kt);
          }
#pragma unroll
          for (int kk = 0; kk < C::KL; ++kk) ktop[kk] = acc_op<T>(kt, kk);
        } else {
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks)
            ktop[ks] = load_rows_op<T>(kb + col, kstride, ks, hh, L, false);
        }
      }
    }
    const float gdl = ka.gd[((size_t)u * ka.nblk + blk) * kTile + li];

    lds_barrier();  // the previous block's LDS readers are done
    float vq[FM::PPW][16], vk[FM::PPW][16];
    FM::logits(wop, qop, w, li, hh, vq, sh.fq);
    if (!delta) FM::logits(wop, kop, w, li, hh, vk, sh.fk);
    lds_barrier();
    FM::exps(w, li, hh, vq, sh.fq);
    if (!delta) FM::exps(w, li, hh, vk, sh.fk);
    lds_barrier();
    FM::scale(w, li, vq, sh.fq);
    if (!delta) FM::scale(w, li, vk, sh.fk);
#pragma unroll
    for (int j = 0; j < RPW; ++j) {
      const int p = w + j * NW;
      if (p >= NRT) continue;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = p * kTile + row_of(i, hh);
        const float x = row_ok ? vq[j][i] : 0.0f;
        const T hi = from_f32<T>(x);
        sh.phiQT[0][r][li] = hi;
        if constexpr (C::NPART == 2) sh.phiQT[1][r][li] = from_f32<T>(x - to_f32(hi));
      }
    }
    if (w == 0 && hh == 0) sh.gd[li] = gdl;

    float dphi[RPW][16];
    if (!delta) {
      // dL/dphi(k_t) = Gbar v_t + gz, with Gbar over the later blocks only.
#pragma unroll
      for (int j = 0; j < RPW; ++j) {
        const int p = w + j * NW;
        if (p >= NRT) continue;
        f32x16 dk = {};
#pragma unroll
        for (int s = 0; s < NW; ++s)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks)
          {
            dk = M::mma(acc_op<T>(gacc[j][s], ks), vrow[s][ks], dk);
            if constexpr (C::NPART == 2) dk = M::mma(acc_op_lo<T>(gacc[j][s], ks), vrow[s][ks], dk);
          }
        float js = 0.0f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          dphi[j][i] = dk[i] + sh.gz[p * kTile + row_of(i, hh)];
          js += dphi[j][i] * vk[j][i];
        }
        js += xor32(js);
        if (hh == 0) sh.jsum[p][li] = js;
      }
      if constexpr (IN) {
        // Gbar^T (before this block's queries join it) and phi(K) to LDS as
        // operand pairs, for dL/dv_t += Gbar^T phi(k_t) below
#pragma unroll
        for (int j = 0; j < RPW; ++j) {
          const int p = w + j * NW;
          if (p >= NRT) continue;
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int r = p * kTile + row_of(i, hh);
            const float x = row_ok ? vk[j][i] : 0.0f;
            const T xh = from_f32<T>(x);
            shi.phiK[0][li][r] = xh;
            if constexpr (C::NPART == 2) shi.phiK[1][li][r] = from_f32<T>(x - to_f32(xh));
#pragma unroll
            for (int s = 0; s < NW; ++s) {
              const float gv = gacc[j][s][i];
              const T gh = from_f32<T>(gv);
              shi.gT[0][s * kTile + row_of(i, hh)][p * kTile + li] = gh;
              if constexpr (C::NPART == 2)
                shi.gT[1][s * kTile + row_of(i, hh)][p * kTile + li] = from_f32<T>(gv - to_f32(gh));
            }
          }
        }
      }
    }
    lds_barrier();
    if constexpr (IN) {
      if (!delta) {
        // dL/dv_t (state part) = Gbar^T phi(k_t): rows c of slice w,
        // columns t; both operands as hi + lo pairs on the bf16 path
        f32x16 dvacc = {};
#pragma unroll
        for (int ks = 0; ks < f / KW; ++ks) {
          const op_t ah = load_op<T>(&shi.gT[0][w * kTile + li][ks * KW + hh * E]);
          const op_t bh = load_op<T>(&shi.phiK[0][li][ks * KW + hh * E]);
          dvacc = M::mma(ah, bh, dvacc);
          if constexpr (C::NPART == 2) {
            dvacc = M::mma(load_op<T>(&shi.gT[1][w * kTile + li][ks * KW + hh * E]), bh, dvacc);
            dvacc = M::mma(ah, load_op<T>(&shi.phiK[1][li][ks * KW + hh * E]), dvacc);
          }
        }
        if (row_ok) {
          float* dst = ka.dvl + ((size_t)u * T_ + t0 + li) * D + w * kTile;
#pragma unroll
          for (int i = 0; i < 16; i += 4)
            *reinterpret_cast<f32x4*>(dst + row_of(i, hh)) =
                f32x4{dvacc[i], dvacc[i + 1], dvacc[i + 2], dvacc[i + 3]};
        }
      }
    }
    if (!delta) {
#pragma unroll
      for (int j = 0; j < RPW; ++j) {
        const int p = w + j * NW;
        if (p >= NRT) continue;
        const int sg = p / NT, t = p % NT;
        float ssum = 0.0f;
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) ssum += sh.jsum[sg * NT + tt][li];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float du = row_ok ? vk[j][i] * (dphi[j][i] - ssum) : 0.0f;
          if (sg) du = -du;
          const int jr = t * kTile + row_of(i, hh);
          const T hi = from_f32<T>(du);
          sh.duT[sg][0][jr][li] = hi;
          if constexpr (C::NPART == 2) sh.duT[sg][1][jr][li] = from_f32<T>(du - to_f32(hi));
        }
      }
    }
    // gz += sum_i phi(q_i) dL/dD_i (gz is not read again in this block).
    for (int r = tid; r < f; r += blockDim.x) {
      float s = 0.0f;
#pragma unroll
      for (int part = 0; part < C::NPART; ++part)
        for (int i = 0; i < kTile; ++i) s += to_f32(sh.phiQT[part][r][i]) * sh.gd[i];
      sh.gz[r] += s;
    }
    // Gbar^T += dL/dN^T phi(Q): rows c of slice s, columns of tile p; the
    // query index runs in natural order on both operands.
#pragma unroll
    for (int j = 0; j < RPW; ++j) {
      const int p = w + j * NW;
      if (p >= NRT) continue;
#pragma unroll
      for (int s = 0; s < NW; ++s)
#pragma unroll
        for (int ks = 0; ks < C::KL; ++ks) {
          op_t gh, gl;
          load_split_op<T>(gnT + (size_t)(s * kTile + li) * kTile + ks * KW + hh * E, gh, gl);
          const op_t ph = load_op<T>(&sh.phiQT[0][p * kTile + li][ks * KW + hh * E]);
          gacc[j][s] = M::mma(gh, ph, gacc[j][s]);
          if constexpr (C::NPART == 2) {
            gacc[j][s] = M::mma(gl, ph, gacc[j][s]);
            gacc[j][s] = M::mma(gh, load_op<T>(&sh.phiQT[1][p * kTile + li][ks * KW + hh * E]),
                                gacc[j][s]);
          }
        }
    }
    if (!delta) {
      lds_barrier();
      if constexpr (IN) {
        // dL/du of the block's keys, both signs summed, for dL/dk = W dL/du
        float* dst = ka.duk + ((size_t)u * T_ + t0) * F;
        for (int it = tid; it < L * (F / 4); it += blockDim.x) {
          const int t = it / (F / 4), j4 = (it % (F / 4)) * 4;
          f32x4 x;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float acc = 0.0f;
#pragma unroll
            for (int sg = 0; sg < 2; ++sg)
#pragma unroll
              for (int part = 0; part < C::NPART; ++part) acc += to_f32(sh.duT[sg][part][j4 + e][t]);
            x[e] = acc;
          }
          *reinterpret_cast<f32x4*>(dst + (size_t)t * F + j4) = x;
        }
      }
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int sg = 0; sg < 2; ++sg)
#pragma unroll
          for (int part = 0; part < C::NPART; ++part)
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks)
              dwacc[t] = M::mma(lds_op_perm<T>(&sh.duT[sg][part][t * kTile + li][0], ks, hh, 0),
                                ktop[ks], dwacc[t]);
    }
  }

  if (delta) {
    float* dst = ka.dG + ((size_t)u * ka.npc + seg) * D * f;
#pragma unroll
    for (int j = 0; j < RPW; ++j) {
      const int p = w + j * NW;
      if (p >= NRT) continue;
#pragma unroll
      for (int s = 0; s < NW; ++s)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          dst[(size_t)(s * kTile + row_of(i, hh)) * f + p * kTile + li] = gacc[j][s][i];
    }
    lds_barrier();
    float* zd = ka.dgz + ((size_t)u * ka.npc + seg) * f;
    for (int r = tid; r < f; r += blockDim.x) zd[r] = sh.gz[r];
  } else {
    float* dwk = ka.dwk + ((size_t)u * nseg + seg) * F * D;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) dwk[(size_t)(t * kTile + row_of(i, hh)) * D + col] = dwacc[t][i];
  }
}


// ---------------------------------------------------------------------------
// 3'. Pipelined reverse delta (bf16, F <= 64): the sum over a segment's
// blocks of phi(Q)^T dL/dN (and phi(Q)^T dL/dD), two blocks per step.
// Waves 0 and 1 compute phi(Q) of the pair's blocks (the whole feature map in
// one wave) and store it transposed as packed hi/lo pairs; waves 2 and 3 turn
// the blocks' dL/dN^T rows (fp32, from the forward walk) into hi/lo
// operands; the state waves accumulate Gbar (rows: features, columns
// 32w..32w+31) with three products per pair of operand pairs.  One barrier
// per block pair; buffers double-buffered.
// ---------------------------------------------------------------------------
template <int D, int F>
struct GDeltaCfg {
  typedef Mma<bf16> M;
  typedef typename M::op_t op_t;
  static constexpr int NC = D / kTile;   // state waves
  static constexpr int NP = 4;           // 2 feature-map + 2 operand waves
  static constexpr int NWAVE = NP + NC;
  static constexpr int f = 2 * F;
  static constexpr int NRT = f / kTile;
  static constexpr int KD = D / M::KW;
  static constexpr int KL = kTile / M::KW;
  typedef WaveFeatMap<bf16, D, F> WFM;
  struct alignas(16) Buf {
    uint32_t phiQT[2][f][kTile + 4];     // per block of the pair: bf16 hi | lo << 16
    op_t gn[2][2][NC][KL][kWave];        // per block: hi/lo, column tile, k-step, lane
    float gd[2][kTile];
  };
  struct alignas(16) Smem {
    Buf buf[2];
    float gz[f];
  };
};

template <int D>
constexpr int gdelta_threads() {
  return kWave * (4 + D / kTile);
}

template <int D, int F>
__global__ __launch_bounds__(gdelta_threads<D>()) void hyb_bwd_gdelta_kernel(BwdKArgs ka) {
  typedef GDeltaCfg<D, F> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  typedef typename C::WFM WFM;
  constexpr int f = C::f, E = M::E, KW = M::KW, NP = C::NP, NC = C::NC;
  static_assert(gdelta_threads<D>() == kWave * C::NWAVE, "launch bounds match the waves");
  __shared__ typename C::Smem sh;
  const BackwardArgs& a = ka.a;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, L = a.s.L, T_ = a.T;
  const int units = a.s.B * Hq, nseg = ka.nseg;
  // pieces of segments 1 .. nseg-1 (segment 0's sum is never needed)
  const int vix = xcd_unit(blockIdx.x, units * ka.npc);
  const int u = vix % units, pc = vix / units;
  const int b = u / Hq, h = u % Hq;
  const size_t qstride = (size_t)Hq * D;
  int blk0, blk1;
  rev_piece(ka, pc, blk0, blk1);
  const int npair = (blk1 - blk0 + 1) / 2;
  const bool row_ok = li < L;
  const int lrow = min(li, L - 1);
  for (int r = tid; r < f; r += blockDim.x) sh.gz[r] = 0.0f;
  lds_barrier();

  if (w < 2) {
    // ---- phi(Q) of block blk0 + 2j + w ----
    const bf16* __restrict__ Wt_h = (const bf16*)a.W + (size_t)h * F * D;
    op_t wop[WFM::NT][C::KD];
    WFM::load_w(Wt_h, li, hh, wop);
    op_t x[C::KD];
    auto load = [&](int blk) {
      const bf16* row = (const bf16*)a.q + (((size_t)b * T_ + (size_t)blk * L) * Hq + h) * D +
                        (size_t)lrow * qstride + hh * E;
#pragma unroll
      for (int ks = 0; ks < C::KD; ++ks) x[ks] = load_op<bf16>(row + ks * KW);
    };
    if (blk0 + w < blk1) load(blk0 + w);
    for (int j = 0; j <= npair; ++j) {
      const int blk = blk0 + 2 * j + w;
      if (j < npair && blk < blk1) {
        typename C::Buf& B = sh.buf[j & 1];
        // a padding row reads row L-1 (finite); keep = row_ok zeroes its phi
        float phi[WFM::NPAIR][16];
        WFM::logits(wop, x, phi);
        if (blk + 2 < blk1) load(blk + 2);  // next pair's block in flight
        WFM::softmax(phi, row_ok);
#pragma unroll
        for (int p = 0; p < WFM::NPAIR; ++p)
#pragma unroll
          for (int i = 0; i < 16; i += 2)
            pack_hi_lo2(phi[p][i], phi[p][i + 1], B.phiQT[w][WFM::feature(16 * p + i, hh)][li],
                        B.phiQT[w][WFM::feature(16 * p + i + 1, hh)][li]);
      }
      lds_barrier();
    }
  } else if (w < NP) {
    // ---- dL/dN^T operands (and dL/dD) of block blk0 + 2j + (w - 2) ----
    // Operand of column tile ct, k-step ks: lane (li, hh) holds column
    // 32ct + li at the block's tokens row_of(ks*E + e, hh) (two runs of 4).
    const int q = w - 2;
    for (int j = 0; j <= npair; ++j) {
      const int blk = blk0 + 2 * j + q;
      if (j < npair && blk < blk1) {
        typename C::Buf& B = sh.buf[j & 1];
        const float* gnT = ka.gnT + ((size_t)u * ka.nblk + blk) * D * kTile;
#pragma unroll
        for (int ct = 0; ct < NC; ++ct)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) {
            const float* src = gnT + (size_t)(ct * kTile + li) * kTile + 16 * ks + 4 * hh;
            const f32x4 x0 = *reinterpret_cast<const f32x4*>(src);
            const f32x4 x1 = *reinterpret_cast<const f32x4*>(src + 8);
            const float xv[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
            op_t hi, lo;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              hi[e] = (bf16)xv[e];
              lo[e] = (bf16)(xv[e] - (float)hi[e]);
            }
            B.gn[q][0][ct][ks][lane] = hi;
            B.gn[q][1][ct][ks][lane] = lo;
          }
        if (lane < kTile) B.gd[q][lane] = ka.gd[((size_t)u * ka.nblk + blk) * kTile + lane];
      }
      lds_barrier();
    }
  } else {
    // ---- state waves: Gbar (features x columns 32cw..) += phi(Q)^T dL/dN ----
    const int cw = w - NP, col = cw * kTile + li;
    f32x16 gacc[C::NRT];
#pragma unroll
    for (int rt = 0; rt < C::NRT; ++rt) gacc[rt] = f32x16{};
    lds_barrier();  // step 0 (peeled: the producers fill the first buffer)
    for (int j = 1; j <= npair; ++j) {
      const int pj = j - 1;
      {
        typename C::Buf& B = sh.buf[pj & 1];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          if (blk0 + 2 * pj + q >= blk1) continue;  // uniform
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) {
            const op_t gh = B.gn[q][0][cw][ks][lane], gl = B.gn[q][1][cw][ks][lane];
#pragma unroll
            for (int rt = 0; rt < C::NRT; ++rt) {
              op_t ph, pl;
              lds_pair_op(&B.phiQT[q][rt * kTile + li][0], ks, hh, ph, pl);
              gacc[rt] = M::mma(ph, gh, gacc[rt]);
              gacc[rt] = M::mma(pl, gh, gacc[rt]);
              gacc[rt] = M::mma(ph, gl, gacc[rt]);
            }
          }
          // gz += sum_i phi(q_i) dL/dD_i
          for (int r = tid - NP * kWave; r < f; r += NC * kWave) {
            float s = 0.0f;
#pragma unroll
            for (int t0 = 0; t0 < kTile; t0 += 4) {
              const uint4 xq = *reinterpret_cast<const uint4*>(&B.phiQT[q][r][t0]);
#pragma unroll
              for (int e = 0; e < 4; ++e)
                s += (unpack_hi(xq[e]) + unpack_lo(xq[e])) * B.gd[q][t0 + e];
            }
            sh.gz[r] += s;
          }
        }
      }
      lds_barrier();
    }
    // Gbar^T tiles as the reverse walk reads them: element (c, r) at c*f + r
    float* dst = ka.dG + ((size_t)u * ka.npc + pc) * D * f;
#pragma unroll
    for (int rt = 0; rt < C::NRT; ++rt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        *reinterpret_cast<f32x4*>(dst + (size_t)col * f + rt * kTile + row_of(4 * jj, hh)) =
            f32x4{gacc[rt][4 * jj], gacc[rt][4 * jj + 1], gacc[rt][4 * jj + 2], gacc[rt][4 * jj + 3]};
    float* zd = ka.dgz + ((size_t)u * ka.npc + pc) * f;
    for (int r = tid - NP * kWave; r < f; r += NC * kWave) zd[r] = sh.gz[r];
  }
}


// ---------------------------------------------------------------------------
// 4'. Pipelined reverse walk (bf16, F <= 64).  Blocks are taken last to
// first; producers prepare block c-1 while the state waves finish block c:
//   wave 0: phi(Q) of the block, stored transposed as packed hi/lo pairs
//           (the operand of the Gbar update);
//   wave 1: phi(K), fp32 [token][feature] (the feature-map Jacobian);
//   wave 2: the V rows as operands of dL/dphi(K) and the K^T operands of dW;
//   wave 3: the dL/dN^T hi/lo operands and dL/dD of the block;
//   state waves (D/32): dL/dphi(K) = Gbar v + gz for the feature tiles they
//           own, the per-sign sums, dL/du (packed hi/lo, transposed), then
//           the Gbar and gz updates, then dW += dL/du^T K for columns
//           32w..32w+31.  Gbar^T and the partial dW stay in registers.
// Two barriers per block (all waves take part): after the per-sign partial
// sums and after dL/du.  No end-of-step barrier: the state waves take the
// block's last operands from the buffer (K^T) before the second barrier, and
// the producers refill it only after that barrier; dL/du is rewritten only
// after the next first barrier, which the state waves reach after their dW.
// ---------------------------------------------------------------------------
template <int D, int F>
struct RWalkCfg {
  typedef Mma<bf16> M;
  typedef typename M::op_t op_t;
  static constexpr int NC = D / kTile;       // state waves / column slices
  static constexpr int NP = 4;
  static constexpr int NWAVE = NP + NC;
  static constexpr int f = 2 * F;
  static constexpr int NRT = f / kTile;      // feature tiles
  static constexpr int NT = F / kTile;       // tiles per sign
  static constexpr int RPW = (NRT + NC - 1) / NC;
  static constexpr int KD = D / M::KW;
  static constexpr int KL = kTile / M::KW;
  typedef WaveFeatMap<bf16, D, F> WFM;
  struct alignas(16) Buf {
    uint32_t phiQT[f][kTile + 4];    // phi(q_i)[r] at [r][i], bf16 hi | lo << 16
    float phiK[kTile][f + 4];        // phi(k_t)[r] at [t][r]
    op_t vrow[NC][KL][kWave];        // V rows: lane (t, hh), columns 32s + row_of
    op_t ktop[NC][KL][kWave];        // K^T: lane (c, hh), tokens in row_of order
    op_t gn[2][NC][KL][kWave];       // dL/dN^T hi, lo: lane (c, hh), tokens natural
    float gd[kTile];
  };
  struct alignas(16) Smem {
    Buf buf[2];
    uint32_t duT[2][F][kTile + 4];   // +-dL/du of each sign at [j][t], packed hi/lo
    float jsum[NRT][kTile];
  };
};

template <int D>
constexpr int rwalk_threads() {
  return kWave * (4 + D / kTile);
}

template <int D, int F>
__global__ __launch_bounds__(rwalk_threads<D>()) void hyb_bwd_rwalk_kernel(BwdKArgs ka) {
  typedef RWalkCfg<D, F> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  typedef typename C::WFM WFM;
  constexpr int f = C::f, E = M::E, KW = M::KW, NP = C::NP, NC = C::NC;
  constexpr int NRT = C::NRT, NT = C::NT, RPW = C::RPW;
  static_assert(rwalk_threads<D>() == kWave * C::NWAVE, "launch bounds match the waves");
  __shared__ typename C::Smem sh;
  const BackwardArgs& a = ka.a;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L, T_ = a.T;
  const int units = a.s.B * Hq, nseg = ka.nseg;
  const int vix = xcd_unit(blockIdx.x, units * nseg);
  const int u = vix % units, seg = vix / units;
  const int b = u / Hq, h = u % Hq, g = h / (Hq / Hkv);
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
  const int blk0 = seg * ka.seg_blocks, blk1 = min(ka.nblk, blk0 + ka.seg_blocks);
  const int nb = blk1 - blk0;
  const bool row_ok = li < L;
  const int lrow = min(li, L - 1);
  auto blk_of = [&](int n) { return blk1 - 1 - n; };  // step n handles block blk_of(n)
  auto qrow = [&](int blk) {
    return (const bf16*)a.q + (((size_t)b * T_ + (size_t)blk * L) * Hq + h) * D;
  };
  auto krow = [&](int blk) {
    return (const bf16*)a.k + (((size_t)b * T_ + (size_t)blk * L) * Hkv + g) * D;
  };
  auto vrowp = [&](int blk) {
    return (const bf16*)a.v + (((size_t)b * T_ + (size_t)blk * L) * Hkv + g) * D;
  };

  lds_barrier();

  if (w < 2) {
    // ---- feature map of Q (wave 0) or K (wave 1) ----
    const bf16* __restrict__ Wt_h = (const bf16*)a.W + (size_t)h * F * D;
    op_t wop[WFM::NT][C::KD];
    WFM::load_w(Wt_h, li, hh, wop);
    op_t x[C::KD];
    auto load = [&](int blk) {
      const bf16* row = (w == 0 ? qrow(blk) + (size_t)lrow * qstride : krow(blk) + (size_t)lrow * kstride) + hh * E;
#pragma unroll
      for (int ks = 0; ks < C::KD; ++ks) x[ks] = load_op<bf16>(row + ks * KW);
    };
    if (nb > 0) load(blk_of(0));
    for (int n = 0; n <= nb; ++n) {
      if (n < nb) {
        typename C::Buf& B = sh.buf[n & 1];
        // a padding row reads row L-1 (finite); keep = row_ok zeroes its phi
        float phi[WFM::NPAIR][16];
        WFM::logits(wop, x, phi);
        if (n + 1 < nb) load(blk_of(n + 1));
        WFM::softmax(phi, row_ok);
        if (w == 0) {
#pragma unroll
          for (int p = 0; p < WFM::NPAIR; ++p)
#pragma unroll
            for (int i = 0; i < 16; i += 2)
              pack_hi_lo2(phi[p][i], phi[p][i + 1], B.phiQT[WFM::feature(16 * p + i, hh)][li],
                          B.phiQT[WFM::feature(16 * p + i + 1, hh)][li]);
        } else {
#pragma unroll
          for (int p = 0; p < WFM::NPAIR; ++p)
#pragma unroll
            for (int i = 0; i < 16; i += 4)
              *reinterpret_cast<f32x4*>(&B.phiK[li][WFM::feature(16 * p + i, hh)]) =
                  f32x4{phi[p][i], phi[p][i + 1], phi[p][i + 2], phi[p][i + 3]};
        }
      }
      lds_barrier();
      lds_barrier();
    }
  } else if (w == 2) {
    // ---- V rows (operands of dL/dphi(K)) and K^T (operands of dW) ----
    op_t vr[NC][C::KL], kt[NC][C::KL];
    auto load = [&](int blk) {
      const bf16* vb = vrowp(blk) + (size_t)lrow * kstride;
#pragma unroll
      for (int s = 0; s < NC; ++s)
#pragma unroll
        for (int ks = 0; ks < C::KL; ++ks) {
          vr[s][ks] = keep_if<bf16>(row_ok, lds_op_perm<bf16>(vb, ks, hh, s * kTile));
          kt[s][ks] = load_rows_op<bf16>(krow(blk) + s * kTile + li, kstride, ks, hh, L, false);
        }
    };
    if (nb > 0) load(blk_of(0));
    for (int n = 0; n <= nb; ++n) {
      if (n < nb) {
        typename C::Buf& B = sh.buf[n & 1];
#pragma unroll
        for (int s = 0; s < NC; ++s)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) {
            B.vrow[s][ks][lane] = vr[s][ks];
            B.ktop[s][ks][lane] = kt[s][ks];
          }
        if (n + 1 < nb) load(blk_of(n + 1));
      }
      lds_barrier();
      lds_barrier();
    }
  } else if (w == 3) {
    // ---- dL/dN^T hi/lo operands (tokens natural) and dL/dD ----
    f32x4 graw[NC][C::KL][2];
    float gdv = 0.0f;
    auto load = [&](int blk) {
      const float* gnT = ka.gnT + ((size_t)u * ka.nblk + blk) * D * kTile;
#pragma unroll
      for (int s = 0; s < NC; ++s)
#pragma unroll
        for (int ks = 0; ks < C::KL; ++ks) {
          const float* src = gnT + (size_t)(s * kTile + li) * kTile + ks * KW + hh * E;
          graw[s][ks][0] = *reinterpret_cast<const f32x4*>(src);
          graw[s][ks][1] = *reinterpret_cast<const f32x4*>(src + 4);
        }
      if (lane < kTile) gdv = ka.gd[((size_t)u * ka.nblk + blk) * kTile + lane];
    };
    if (nb > 0) load(blk_of(0));
    for (int n = 0; n <= nb; ++n) {
      if (n < nb) {
        typename C::Buf& B = sh.buf[n & 1];
#pragma unroll
        for (int s = 0; s < NC; ++s)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) {
            op_t gh, gl;
            split_op(graw[s][ks][0], graw[s][ks][1], gh, gl);
            B.gn[0][s][ks][lane] = gh;
            B.gn[1][s][ks][lane] = gl;
          }
        if (lane < kTile) B.gd[lane] = gdv;
        if (n + 1 < nb) load(blk_of(n + 1));
      }
      lds_barrier();
      lds_barrier();
    }
  } else {
    // ---- state waves ----
    const int cw = w - NP, col = cw * kTile + li;
    // Gbar^T tiles (rows c of slice s, columns of feature tile p): the sums
    // over the later segments
    // (the first increment straight into the accumulators, as in the
    // forward walk)
    f32x16 gacc[RPW][NC];
#pragma unroll
    for (int j = 0; j < RPW; ++j)
#pragma unroll
      for (int s = 0; s < NC; ++s) gacc[j][s] = f32x16{};
    auto add_increment = [&](int sp, bool first) {
      const float* src = ka.dG + ((size_t)u * ka.npc + sp) * D * f;
#pragma unroll
      for (int j = 0; j < RPW; ++j) {
        const int p = cw + j * NC;
        if (p >= NRT) continue;
#pragma unroll
        for (int s = 0; s < NC; ++s)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const float y = src[(size_t)(s * kTile + row_of(i, hh)) * f + p * kTile + li];
            gacc[j][s][i] = first ? y : gacc[j][s][i] + y;
          }
      }
    };
    if (seg * ka.ppseg < ka.npc) add_increment(seg * ka.ppseg, true);
    for (int sp = seg * ka.ppseg + 1; sp < ka.npc; ++sp) add_increment(sp, false);
    // gz for the same feature tiles, as accumulator tiles whose columns are
    // all equal (register i: feature 32p + row_of(i, hh)); its update
    // phi(Q)^T dL/dD runs on the MFMAs against a broadcast dL/dD operand
    f32x16 gzt[RPW];
#pragma unroll
    for (int j = 0; j < RPW; ++j) {
      gzt[j] = f32x16{};
      const int p = cw + j * NC;
      if (p >= NRT) continue;
      for (int sp = seg * ka.ppseg; sp < ka.npc; ++sp)
#pragma unroll
        for (int i = 0; i < 16; ++i) gzt[j][i] += ka.dgz[((size_t)u * ka.npc + sp) * f + p * kTile + row_of(i, hh)];
    }
    f32x16 dwacc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) dwacc[t] = f32x16{};
    // step 0: the producers fill the first buffer
    lds_barrier();
    lds_barrier();
    for (int n = 1; n <= nb; ++n) {
      {
        typename C::Buf& B = sh.buf[(n - 1) & 1];
        // dL/dphi(k_t) = Gbar v_t + gz (Gbar over the later blocks only)
        float dphi[RPW][16], pk[RPW][16];
#pragma unroll
        for (int j = 0; j < RPW; ++j) {
          const int p = cw + j * NC;
          if (p >= NRT) continue;
          f32x16 dk = {};
#pragma unroll
          for (int s = 0; s < NC; ++s)
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks) {
              const op_t vb = B.vrow[s][ks][lane];
              op_t gh, gl;
              acc_op_pair(gacc[j][s], ks, gh, gl);
              dk = M::mma(gh, vb, dk);
              dk = M::mma(gl, vb, dk);
            }
          float js = 0.0f;
#pragma unroll
          for (int i4 = 0; i4 < 16; i4 += 4) {
            const int r = p * kTile + row_of(i4, hh);
            const f32x4 pk4 = *reinterpret_cast<const f32x4*>(&B.phiK[li][r]);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              pk[j][i4 + e] = pk4[e];
              dphi[j][i4 + e] = dk[i4 + e] + gzt[j][i4 + e];
              js += dphi[j][i4 + e] * pk4[e];
            }
          }
          js += xor32(js);
          if (hh == 0) sh.jsum[p][li] = js;
        }
        lds_barrier();
        // dL/du for each sign, transposed and packed (phi(k) of a padding
        // token is stored as zero, so is its dL/du)
#pragma unroll
        for (int j = 0; j < RPW; ++j) {
          const int p = cw + j * NC;
          if (p >= NRT) continue;
          const int sg = p / NT, t = p % NT;
          float ssum = 0.0f;
#pragma unroll
          for (int tt = 0; tt < NT; ++tt) ssum += sh.jsum[sg * NT + tt][li];
          const float sgn = sg ? -1.0f : 1.0f;
#pragma unroll
          for (int i = 0; i < 16; i += 2)
            pack_hi_lo2(sgn * pk[j][i] * (dphi[j][i] - ssum), sgn * pk[j][i + 1] * (dphi[j][i + 1] - ssum),
                        sh.duT[sg][t * kTile + row_of(i, hh)][li],
                        sh.duT[sg][t * kTile + row_of(i + 1, hh)][li]);
        }
        // dL/dD of the block's queries (natural order) as a broadcast operand
        // pair: gz += phi(Q)^T dL/dD below (every read of gz this step is above)
        op_t gdh[C::KL], gdl[C::KL];
#pragma unroll
        for (int ks = 0; ks < C::KL; ++ks)
          split_op(*reinterpret_cast<const f32x4*>(&B.gd[ks * KW + hh * E]),
                   *reinterpret_cast<const f32x4*>(&B.gd[ks * KW + hh * E + 4]), gdh[ks], gdl[ks]);
        // Gbar^T += dL/dN^T phi(Q) (rows c of slice s, columns of tile p)
#pragma unroll
        for (int j = 0; j < RPW; ++j) {
          const int p = cw + j * NC;
          if (p >= NRT) continue;
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) {
            op_t ph, pl;
            lds_pair_op_nat(&B.phiQT[p * kTile + li][0], ks, hh, ph, pl);
            gzt[j] = M::mma(ph, gdh[ks], gzt[j]);
            gzt[j] = M::mma(pl, gdh[ks], gzt[j]);
            gzt[j] = M::mma(ph, gdl[ks], gzt[j]);
#pragma unroll
            for (int s = 0; s < NC; ++s) {
              const op_t gh = B.gn[0][s][ks][lane], gl = B.gn[1][s][ks][lane];
              gacc[j][s] = M::mma(gh, ph, gacc[j][s]);
              gacc[j][s] = M::mma(gl, ph, gacc[j][s]);
              gacc[j][s] = M::mma(gh, pl, gacc[j][s]);
              __builtin_amdgcn_sched_barrier(0);  // keep operand reads near their use
            }
          }
        }
        // the K^T operands of dW, read before the barrier: the producers
        // refill this buffer right after it
        op_t kb[C::KL];
#pragma unroll
        for (int ks = 0; ks < C::KL; ++ks) kb[ks] = B.ktop[cw][ks][lane];
        lds_barrier();
        // dW^T tiles (rows j of tile t, columns 32cw..) += dL/du^T K
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int sg = 0; sg < 2; ++sg)
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks) {
              op_t uh, ul;
              lds_pair_op(&sh.duT[sg][t * kTile + li][0], ks, hh, uh, ul);
              dwacc[t] = M::mma(uh, kb[ks], dwacc[t]);
              dwacc[t] = M::mma(ul, kb[ks], dwacc[t]);
              __builtin_amdgcn_sched_barrier(0);
            }
      }
    }
    float* dwk = ka.dwk + ((size_t)u * nseg + seg) * F * D;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) dwk[(size_t)(t * kTile + row_of(i, hh)) * D + col] = dwacc[t][i];
  }
}

// ---------------------------------------------------------------------------
// 6. Gradients with respect to the inputs q, k, v.  With a_ij = exp(s_ij),
// s_ij = q_i . k_j / sqrt(d) for i, j in one block, and dL/dN, dL/dD from the
// forward walk:
//   dL/ds_ij = w a_ij (dL/dN_i . v_j + dL/dD_i)
//   dL/dq_i  = sum_j dL/ds_ij k_j / sqrt(d) + W_h dL/du(q_i)
//   dL/dk_j  = sum_h [ sum_i dL/ds_ij q_i / sqrt(d) + W_h dL/du(k_j) ]
//   dL/dv_j  = sum_h [ sum_i w a_ij dL/dN_i + Gbar_c^T phi(k_j) ]
// where dL/du(q), dL/du(k) and Gbar^T phi(k) come from the walks.  Blocks are
// independent: one workgroup per (request, KV head, block), NW = D/32 waves,
// wave w forming columns 32w .. 32w+31 of every output; the G query heads of
// the KV head run in turn and dk, dv sum over them in registers.  The 32x32
// score and dL/dP tiles are formed in both orientations (queries in lanes for
// dq, keys in lanes for dk and dv), so each feeds its product straight from
// the accumulators.  w a_ij is evaluated as exp(log w + s_ij): scores must
// stay well inside the fp32 exponent range (the forward walk's 1/D has the
// same limit).
// ---------------------------------------------------------------------------
template <typename T, int D, int F>
struct InCfg {
  typedef Mma<T> M;
  typedef typename M::op_t op_t;
  static constexpr int NW = D / kTile;
  static constexpr int NPART = sizeof(T) == 2 ? 2 : 1;
  static constexpr int PAD = 16 / (int)sizeof(T);
  static constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16 bytes
  static constexpr int KD = D / M::KW;
  static constexpr int KL = kTile / M::KW;
  static constexpr int KF = F / M::KW;
  struct alignas(16) Smem {
    T k[kTile][D + PAD];
    T v[kTile][D + PAD];
    T q[kTile][D + PAD];
    T dn[NPART][kTile][D + PAD];  // dL/dN_i[c] at [part][i][c]
    T wt[F][D + PAD];             // W_h[c][j] at [j][c] (the layout of W)
    float gd[kTile];
  };
};

// An operand whose element e is col[idx(e) * ld]: idx(e) = row_of(ks*E + e,
// hh) (accumulator-row order) or, natural, ks*KW + hh*E + e.
template <typename T>
__device__ inline typename Mma<T>::op_t lds_col_op(const T* col, int ld, int ks, int hh,
                                                   bool natural) {
  typedef Mma<T> M;
  typename M::op_t x;
  if constexpr (M::E == 1) {
    x = col[(size_t)(natural ? ks * M::KW + hh : row_of(ks, hh)) * ld];
  } else {
#pragma unroll
    for (int e = 0; e < M::E; ++e)
      x[e] = col[(size_t)(natural ? ks * M::KW + hh * M::E + e : row_of(ks * M::E + e, hh)) * ld];
  }
  return x;
}

// Accumulator registers ks*E .. as an operand pair hi + lo (lo zero on fp32).
template <typename T>
__device__ inline void acc_split(const f32x16& x, int ks, typename Mma<T>::op_t& hi,
                                 typename Mma<T>::op_t& lo) {
  if constexpr (Mma<T>::E == 1) {
    hi = x[ks];
    lo = 0.0f;
  } else {
    acc_op_pair(x, ks, hi, lo);
  }
}

template <typename T, int D, int F>
__global__ __launch_bounds__(kWave*(D / kTile)) void hyb_bwd_inputs_kernel(BwdKArgs ka) {
  typedef InCfg<T, D, F> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  constexpr int E = M::E, KW = M::KW, EPC = C::EPC, LD = D + C::PAD;
  __shared__ typename C::Smem sh;
  const BackwardArgs& a = ka.a;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L, T_ = a.T, G = Hq / Hkv;
  const int nblk = ka.nblk;
  const int blk = blockIdx.x % nblk, bg = blockIdx.x / nblk;
  const int b = bg / Hkv, g = bg % Hkv;
  const size_t t0 = (size_t)blk * L;
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
  const float scale = 1.0f / sqrtf((float)D);
  const int cc = w * kTile + li;  // this lane's output column
  const bool lrow = li < L;

  // The staging loops below have compile-time trip counts (NTHR threads)
  // and issue all of a thread's loads before its first LDS store: a loop
  // that stores each value as it lands waits a full memory round trip per
  // iteration.
  constexpr int NTHR = kWave * C::NW;
  // rows of a [.][stride] tensor into a [32][LD] LDS tile, rows past L zero
  auto stage_rows = [&](T (*dst)[LD], const T* src, size_t stride) {
    constexpr int N = kTile * (D / EPC) / NTHR;
    static_assert(N * NTHR == kTile * (D / EPC), "whole passes");
    uint4 x[N];
#pragma unroll
    for (int k = 0; k < N; ++k) {
      const int it = tid + k * NTHR, r = it / (D / EPC), c = (it % (D / EPC)) * EPC;
      x[k] = *reinterpret_cast<const uint4*>(src + (size_t)min(r, L - 1) * stride + c);
    }
#pragma unroll
    for (int k = 0; k < N; ++k) {
      const int it = tid + k * NTHR, r = it / (D / EPC), c = (it % (D / EPC)) * EPC;
      *reinterpret_cast<uint4*>(&dst[r][c]) = r < L ? x[k] : uint4{0u, 0u, 0u, 0u};
    }
  };
  stage_rows(sh.k, (const T*)a.k + (((size_t)b * T_ + t0) * Hkv + g) * D, kstride);
  stage_rows(sh.v, (const T*)a.v + (((size_t)b * T_ + t0) * Hkv + g) * D, kstride);

  // A head's staged operands (its Q rows, dL/dN^T, W_h and dL/dD) are
  // fetched into registers while the previous head is computed, then moved
  // to LDS.
  constexpr int NQ = kTile * (D / EPC) / NTHR, NG = D * kTile / NTHR, NWT = F * (D / EPC) / NTHR;
  static_assert(NQ * NTHR == kTile * (D / EPC) && NG * NTHR == D * kTile &&
                    NWT * NTHR == F * (D / EPC),
                "whole passes");
  struct HeadRegs {
    uint4 xq[NQ];
    float xg[NG];
    uint4 xw[NWT];
    float gdl, alpha;
    float xv[16];  // the state part of dv at this lane's rows (below)
  };
  auto fetch = [&](int hq, HeadRegs& r) {
    const int h = g * G + hq;
    const size_t u = (size_t)b * Hq + h;
    const T* qsrc = (const T*)a.q + (((size_t)b * T_ + t0) * Hq + h) * D;
#pragma unroll
    for (int k = 0; k < NQ; ++k) {
      const int it = tid + k * NTHR, rr = it / (D / EPC), c = (it % (D / EPC)) * EPC;
      r.xq[k] = *reinterpret_cast<const uint4*>(qsrc + (size_t)min(rr, L - 1) * qstride + c);
    }
    const float* gn = ka.gnT + (u * nblk + blk) * D * kTile;  // dL/dN^T [c][i]
#pragma unroll
    for (int k = 0; k < NG; ++k) r.xg[k] = gn[tid + k * NTHR];
    const T* wsrc = (const T*)a.W + (size_t)h * F * D;
#pragma unroll
    for (int k = 0; k < NWT; ++k) {
      const int it = tid + k * NTHR, j = it / (D / EPC), c = (it % (D / EPC)) * EPC;
      r.xw[k] = *reinterpret_cast<const uint4*>(wsrc + (size_t)j * D + c);
    }
    r.gdl = tid < kTile ? ka.gd[(u * nblk + blk) * kTile + tid] : 0.0f;
    r.alpha = a.alpha[h];
    // Gbar^T phi(k_j) from the reverse walk, rows j = row_of(r, hh) (rows
    // past the block read row L-1 and are dropped where they are added)
    const float* vsrc = ka.dvl + (u * T_ + t0) * D + cc;
#pragma unroll
    for (int i = 0; i < 16; ++i) r.xv[i] = vsrc[(size_t)min(row_of(i, hh), L - 1) * D];
  };
  auto put = [&](const HeadRegs& r) {
#pragma unroll
    for (int k = 0; k < NQ; ++k) {
      const int it = tid + k * NTHR, rr = it / (D / EPC), c = (it % (D / EPC)) * EPC;
      *reinterpret_cast<uint4*>(&sh.q[rr][c]) = rr < L ? r.xq[k] : uint4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int k = 0; k < NG; ++k) {
      const int it = tid + k * NTHR, c = it / kTile, i = it % kTile;
      const float x = i < L ? r.xg[k] : 0.0f;
      const T xh = from_f32<T>(x);
      sh.dn[0][i][c] = xh;
      if constexpr (C::NPART == 2) sh.dn[1][i][c] = from_f32<T>(x - to_f32(xh));
    }
    if (tid < kTile) sh.gd[tid] = tid < L ? r.gdl : 0.0f;
#pragma unroll
    for (int k = 0; k < NWT; ++k) {
      const int it = tid + k * NTHR, j = it / (D / EPC), c = (it % (D / EPC)) * EPC;
      *reinterpret_cast<uint4*>(&sh.wt[j][c]) = r.xw[k];
    }
  };
  HeadRegs hr;
  fetch(0, hr);

  f32x16 dks = {}, dkl = {}, dva = {};
  for (int hq = 0; hq < G; ++hq) {
    const int h = g * G + hq;
    const size_t u = (size_t)b * Hq + h;
    const float lw = log_sigmoid(hr.alpha);
    float xv[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) xv[i] = hr.xv[i];
    lds_barrier();  // the previous head's readers are done
    put(hr);
    if (hq + 1 < G) fetch(hq + 1, hr);  // the next head's operands in flight
    lds_barrier();

    // Scores and dL/dP = dL/dN_i . v_j: queries in lanes (sq, pq: rows j,
    // columns i) and keys in lanes (sk, pk: rows i, columns j).
    f32x16 sq = {}, sk = {}, pq = {}, pk = {};
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks) {
      const op_t ko = load_op<T>(&sh.k[li][ks * KW + hh * E]);
      const op_t qo = load_op<T>(&sh.q[li][ks * KW + hh * E]);
      const op_t vo = load_op<T>(&sh.v[li][ks * KW + hh * E]);
      const op_t nh = load_op<T>(&sh.dn[0][li][ks * KW + hh * E]);
      sq = M::mma(ko, qo, sq);
      sk = M::mma(qo, ko, sk);
      pq = M::mma(vo, nh, pq);
      pk = M::mma(nh, vo, pk);
      if constexpr (C::NPART == 2) {
        const op_t nl = load_op<T>(&sh.dn[1][li][ks * KW + hh * E]);
        pq = M::mma(vo, nl, pq);
        pk = M::mma(nl, vo, pk);
      }
    }
    // w a_ij and dL/ds_ij in both orientations (zero outside the block)
    f32x16 dsq, ak, dsk;
    {
      const float gdi = sh.gd[li];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int o = row_of(r, hh);
        const float aq = (lrow && o < L) ? expf(lw + sq[r] * scale) : 0.0f;
        dsq[r] = aq * (pq[r] + gdi);
        ak[r] = (lrow && o < L) ? expf(lw + sk[r] * scale) : 0.0f;
        dsk[r] = ak[r] * (pk[r] + sh.gd[o]);
      }
    }

    // dq: sum_j ds_ij k_j (scaled after) + du(q_i) W_h^T
    f32x16 dqs = {}, dql = {};
#pragma unroll
    for (int ks = 0; ks < C::KL; ++ks) {
      op_t hi, lo;
      acc_split<T>(dsq, ks, hi, lo);
      const op_t kc = lds_col_op<T>(&sh.k[0][cc], LD, ks, hh, false);
      dqs = M::mma(hi, kc, dqs);
      if constexpr (C::NPART == 2) dqs = M::mma(lo, kc, dqs);
      // dk (this head): sum_i ds_ij q_i
      acc_split<T>(dsk, ks, hi, lo);
      const op_t qc = lds_col_op<T>(&sh.q[0][cc], LD, ks, hh, false);
      dks = M::mma(hi, qc, dks);
      if constexpr (C::NPART == 2) dks = M::mma(lo, qc, dks);
      // dv (this head): sum_i w a_ij dL/dN_i
      acc_split<T>(ak, ks, hi, lo);
      const op_t nc = lds_col_op<T>(&sh.dn[0][0][cc], LD, ks, hh, false);
      dva = M::mma(hi, nc, dva);
      if constexpr (C::NPART == 2) {
        dva = M::mma(lo, nc, dva);
        dva = M::mma(hi, lds_col_op<T>(&sh.dn[1][0][cc], LD, ks, hh, false), dva);
      }
    }
    // feature-map parts: du (rows: tokens, natural F) times W_h^T
    {
      const float* duq = ka.duq + (u * T_ + t0 + min(li, L - 1)) * F;
      const float* duk = ka.duk + (u * T_ + t0 + min(li, L - 1)) * F;
#pragma unroll
      for (int ks = 0; ks < C::KF; ++ks) {
        const op_t wc = lds_col_op<T>(&sh.wt[0][cc], LD, ks, hh, true);
        op_t hi, lo;
        load_split_op<T>(duq + ks * KW + hh * E, hi, lo);
        hi = keep_if<T>(lrow, hi);
        lo = keep_if<T>(lrow, lo);
        dql = M::mma(hi, wc, dql);
        if constexpr (C::NPART == 2) dql = M::mma(lo, wc, dql);
        load_split_op<T>(duk + ks * KW + hh * E, hi, lo);
        hi = keep_if<T>(lrow, hi);
        lo = keep_if<T>(lrow, lo);
        dkl = M::mma(hi, wc, dkl);
        if constexpr (C::NPART == 2) dkl = M::mma(lo, wc, dkl);
      }
    }
    // dq of head h: rows i (queries), column cc
    {
      float* dst = a.dq + (((size_t)b * T_ + t0) * Hq + h) * D + cc;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = row_of(r, hh);
        if (i < L) dst[(size_t)i * qstride] = dqs[r] * scale + dql[r];
      }
    }
    // the state part of dv: Gbar^T phi(k_j) from the reverse walk
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (row_of(r, hh) < L) dva[r] += xv[r];
  }
  // dk, dv of the KV head: rows j (keys), column cc
  float* dkd = a.dk + (((size_t)b * T_ + t0) * Hkv + g) * D + cc;
  float* dvd = a.dv + (((size_t)b * T_ + t0) * Hkv + g) * D + cc;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int j = row_of(r, hh);
    if (j < L) {
      dkd[(size_t)j * kstride] = dks[r] * scale + dkl[r];
      dvd[(size_t)j * kstride] = dva[r];
    }
  }
}

// ---------------------------------------------------------------------------
// 5. Sum of the partials over requests and segments, in a fixed order.
// ---------------------------------------------------------------------------
__global__ void hyb_bwd_reduce_kernel(BwdKArgs ka) {
  const BackwardArgs& a = ka.a;
  const int Hq = a.s.Hq, F = a.s.F, D = a.s.D, nseg = ka.nseg;
  const size_t per = (size_t)F * D;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx < (size_t)Hq * per) {
    const int h = (int)(idx / per);
    const size_t e = idx % per;
    // terms t = b * nseg + sg in increasing order; each batch's loads are
    // issued before its additions, which keep that order
    const int nterm = a.s.B * nseg;
    constexpr int CH = 8;
    float s = 0.0f;
    for (int t0 = 0; t0 < nterm; t0 += CH) {
      float q[CH], k[CH];
#pragma unroll
      for (int j = 0; j < CH; ++j) {
        const int t = min(t0 + j, nterm - 1);  // in bounds; unused past nterm
        const size_t o = (((size_t)(t / nseg) * Hq + h) * nseg + t % nseg) * per + e;
        q[j] = ka.dwq[o];
        k[j] = ka.dwk[o];
      }
#pragma unroll
      for (int j = 0; j < CH; ++j)
        if (t0 + j < nterm) s += q[j] + k[j];
    }
    a.dW[idx] = s;
  }
  if (idx < (size_t)Hq) {
    float s0 = 0.0f, s1 = 0.0f;
    for (int b = 0; b < a.s.B; ++b) {
      const size_t u = (size_t)b * Hq + idx;
      for (int sg = 0; sg < nseg; ++sg) {
        s0 += ka.red[(u * nseg + sg) * 2];
        s1 += ka.red[(u * nseg + sg) * 2 + 1];
      }
    }
    a.dalpha[idx] = s0;
    if (a.loss) a.loss[idx] = s1;
  }
}

template <typename T, int D, int F>
static hipError_t bwd_go(const BackwardArgs& a, hipStream_t st) {
  const Shape& s = a.s;
  const int units = s.B * s.Hq, nblk = a.T / s.L;
  const SegPlan plan = segment_plan(s, a.T);
  const int nseg = plan.nseg;
  const int seg_blocks = plan.sb;
  const bool inputs = a.dq != nullptr;
  const BwdLayout l = bwd_layout(s, a.T, inputs);
  char* ws = (char*)a.ws;
  const size_t f = 2 * (size_t)s.F;
  BwdKArgs ka;
  ka.a = a;
  ka.nseg = nseg;
  ka.seg_blocks = seg_blocks;
  ka.ppseg = plan.ppseg;
  ka.npc = plan.npieces();
  ka.pb = plan.pb;
  ka.nblk = nblk;
  ka.dS = (float*)(ws + l.dS);
  ka.dz = ka.dS + (size_t)units * ka.npc * s.D * f;
  ka.dG = (float*)(ws + l.dG);
  ka.dgz = (float*)(ws + l.dgz);
  ka.gnT = (float*)(ws + l.gnT);
  ka.gd = (float*)(ws + l.gd);
  ka.dwq = (float*)(ws + l.dwq);
  ka.dwk = (float*)(ws + l.dwk);
  ka.red = (float*)(ws + l.red);
  ka.duq = inputs ? (float*)(ws + l.duq) : nullptr;
  ka.duk = inputs ? (float*)(ws + l.duk) : nullptr;
  ka.dvl = inputs ? (float*)(ws + l.dvl) : nullptr;
  const dim3 block(kWave * (D / kTile));
  hipError_t e;
  if (nseg > 1) {
    // 1. each segment's own state increment (the prefill's delta launch)
    PrefillArgs pa{s, a.T, nullptr, a.k, a.v, a.W, nullptr, nullptr, nullptr,
                   nullptr, nullptr, ka.dS};
    pa.s.n_slots = s.B;
    if ((e = launch_prefill_delta(pa, plan, st)) != hipSuccess) return e;
  }
  // bf16 takes the pipelined forward walk (which also writes dL/du of the
  // queries when the input gradients are asked for); fp32 the four-wave one.
  // The reverse walk with the input gradients is the four-wave one for both
  // dtypes (it also writes dL/du of the keys and Gbar^T phi(K)).
  if constexpr (sizeof(T) == 2) {
    // (the pipelined walk addresses a request's upstream rows and a unit's
    // dL/dN^T through 32-bit buffer offsets)
    const bool fits = (size_t)a.T * s.Hq * D * sizeof(T) < ((size_t)1 << 31) &&
                      (size_t)ka.nblk * D * kTile * sizeof(float) < ((size_t)1 << 31);
    if (fits)
      hipLaunchKernelGGL((hyb_bwd_fpipe_kernel<D, F>), dim3(units * nseg), dim3(fpipe_threads<D>()),
                         0, st, ka);
    else if (inputs)
      hipLaunchKernelGGL((hyb_bwd_fwd_kernel<T, D, F, true>), dim3(units * nseg), block, 0, st, ka);
    else
      hipLaunchKernelGGL((hyb_bwd_fwd_kernel<T, D, F, false>), dim3(units * nseg), block, 0, st, ka);
  } else if (inputs) {
    hipLaunchKernelGGL((hyb_bwd_fwd_kernel<T, D, F, true>), dim3(units * nseg), block, 0, st, ka);
  } else {
    hipLaunchKernelGGL((hyb_bwd_fwd_kernel<T, D, F, false>), dim3(units * nseg), block, 0, st, ka);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (nseg > 1) {
    if constexpr (sizeof(T) == 2) {
      hipLaunchKernelGGL((hyb_bwd_gdelta_kernel<D, F>), dim3(units * ka.npc),
                         dim3(gdelta_threads<D>()), 0, st, ka);
    } else {
      hipLaunchKernelGGL((hyb_bwd_rev_kernel<T, D, F, false>), dim3(units * ka.npc), block, 0,
                         st, ka, 1);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (inputs) {
    hipLaunchKernelGGL((hyb_bwd_rev_kernel<T, D, F, true>), dim3(units * nseg), block, 0, st, ka,
                       0);
  } else if constexpr (sizeof(T) == 2) {
    hipLaunchKernelGGL((hyb_bwd_rwalk_kernel<D, F>), dim3(units * nseg), dim3(rwalk_threads<D>()),
                       0, st, ka);
  } else {
    hipLaunchKernelGGL((hyb_bwd_rev_kernel<T, D, F, false>), dim3(units * nseg), block, 0, st, ka,
                       0);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (inputs) {
    hipLaunchKernelGGL((hyb_bwd_inputs_kernel<T, D, F>), dim3(s.B * s.Hkv * nblk), block, 0, st,
                       ka);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const size_t n = (size_t)s.Hq * s.F * s.D;
  hipLaunchKernelGGL(hyb_bwd_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                     ka);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t bwd_f(const BackwardArgs& a, hipStream_t st) {
  switch (a.s.F) {
    case 32: return bwd_go<T, D, 32>(a, st);
    case 64: return bwd_go<T, D, 64>(a, st);
  }
  return hipErrorInvalidValue;
}

template <typename T>
static hipError_t bwd_d(const BackwardArgs& a, hipStream_t st) {
  switch (a.s.D) {
    case 64: return bwd_f<T, 64>(a, st);
    case 128: return bwd_f<T, 128>(a, st);
  }
  return hipErrorInvalidValue;
}

bool backward_supported(const Shape& s) { return s.F == 32 || s.F == 64; }

hipError_t launch_backward(const BackwardArgs& a, hipStream_t st) {
  return a.s.dtype == 1 ? bwd_d<bf16>(a, st) : bwd_d<float>(a, st);
}

}  // namespace hyb
