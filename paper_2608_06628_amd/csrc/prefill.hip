// prefill.hip -- block-causal prefill of a prompt into the recurrent state
// (Figure 2 pattern): block c is answered against the state of blocks
// 0..c-1 -- exact softmax inside the block, linear readout of the state,
// gated merge (Section 3.1) -- and is then committed,
// S += phi(K_c)^T V_c, z += sum phi(K_c).
//
// Sequence segments.  The prompt's blocks are cut into nseg segments so that
// the grid fills the chip (SegPlan).  A first launch (delta mode) computes the
// state increments dS = sum_c phi(K_c)^T V_c and dz of the blocks of segments
// 0 .. nseg-2, in pieces of a segment each or smaller, into the caller's
// workspace; the second launch (walk mode) starts segment s from S + the
// increments of the pieces before it and walks its blocks as below; the last
// segment writes the final state.  Only the associativity of the sum is used,
// so the result is the sequential one up to rounding order.  Without outputs,
// only the last segment walks.
// Ordering: with nseg > 1 the walk segments start from a snapshot of the
// incoming S, z that a launch before the walk copies into the workspace, never
// from S, z themselves, which the last segment overwrites in the same launch
// (workgroups of one launch are not ordered).
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
#include <type_traits>

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

// Workspace layout (nseg > 1): the increments dS [units][npieces][D][f] and
// dz [units][npieces][f], then the snapshot of the incoming state,
// S0 [units][D][f] and z0 [units][f].
__device__ inline const float* prefill_snapshot_S(const PrefillArgs& a, int npc, int u) {
  const size_t f = 2 * (size_t)a.s.F, units = (size_t)a.s.B * a.s.Hq;
  return a.ws + units * npc * (a.s.D * f + f) + (size_t)u * a.s.D * f;
}
__device__ inline const float* prefill_snapshot_z(const PrefillArgs& a, int npc, int u) {
  const size_t f = 2 * (size_t)a.s.F, units = (size_t)a.s.B * a.s.Hq;
  return a.ws + units * npc * (a.s.D * f + f) + units * a.s.D * f + (size_t)u * f;
}

// Snapshot of the incoming state of every (request, head) unit into the
// workspace, one workgroup per unit, 16-byte copies.  A unit whose slot is
// out of range is skipped (its walk never reads the snapshot).
__global__ __launch_bounds__(256) void hyb_prefill_snapshot_kernel(PrefillArgs a, int npc) {
  const int u = blockIdx.x, Hq = a.s.Hq;
  const int b = u / Hq, h = u % Hq;
  const int slot = a.slots ? a.slots[b] : b;
  if (slot < 0 || slot >= a.s.n_slots) return;
  const size_t f = 2 * (size_t)a.s.F, n = (size_t)a.s.D * f;
  const size_t sbase = (size_t)slot * Hq + h;
  const f32x4* src = reinterpret_cast<const f32x4*>(a.S + sbase * n);
  f32x4* dst = reinterpret_cast<f32x4*>(const_cast<float*>(prefill_snapshot_S(a, npc, u)));
  for (size_t i = threadIdx.x; i < n / 4; i += blockDim.x) dst[i] = src[i];
  float* dz = const_cast<float*>(prefill_snapshot_z(a, npc, u));
  for (size_t i = threadIdx.x; i < f; i += blockDim.x) dz[i] = a.z[sbase * f + i];
}

template <typename T, int D, int F>
__global__ __launch_bounds__(kWave*(D / kTile)) void hyb_prefill_kernel(
    PrefillArgs a, SegPlan p, int delta) {
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
  // (delta mode: one workgroup per (unit, piece); walk mode: per (unit,
  // segment))
  const int units = a.s.B * Hq, nseg = p.nseg, npc = p.npieces();
  const int vix = xcd_unit(blockIdx.x, units * (delta ? npc : nseg));
  const int u = vix % units, seg = vix / units;
  const int b = u / Hq, h = u % Hq, g = h / (Hq / Hkv);
  const int slot = a.slots ? a.slots[b] : b;
  const bool want_out = !delta && a.out != nullptr;
  const bool last = !delta && seg == nseg - 1;
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
  const int col = w * kTile + li;
  const int nblk = T_ / L;
  const int blk0 = delta ? p.piece_lo(seg) : seg * p.sb;
  const int blk1 = min(nblk, delta ? p.piece_hi(seg) : blk0 + p.sb);
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
  // Workspace: dS [units][npieces][D][f] (transposed, as S), then dz
  // [units][npieces][f].
  float* __restrict__ wsS = a.ws + (size_t)u * npc * D * f;
  float* __restrict__ wsz = a.ws + (size_t)units * npc * D * f + (size_t)u * npc * f;
  // (without outputs only the last segment walks, and no snapshot is taken)
  const bool snap = nseg > 1 && a.out != nullptr;
  const float* __restrict__ S0 = snap ? prefill_snapshot_S(a, npc, u) : Sh;
  const float* __restrict__ z0 = snap ? prefill_snapshot_z(a, npc, u) : zh;

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
    add_state(S0, true);
    for (int s = 0; s < seg * p.ppseg; ++s) add_state(wsS + (size_t)s * D * f, false);
    for (int r = tid; r < f; r += blockDim.x) {
      float zr = z0[r];
      for (int s = 0; s < seg * p.ppseg; ++s) zr += wsz[(size_t)s * f + r];
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


// ---------------------------------------------------------------------------
// Pipelined walk (bf16, F <= 64, outputs wanted): one workgroup per (request,
// head, segment), 4 + D/32 waves.  The roles work on different blocks of the
// segment and meet at one barrier per iteration; in iteration it:
//   QS waves (0, 1: even and odd blocks): phi(Q) and the in-block softmax of
//     a block over two iterations -- the logits, the scores, the first
//     exponentials and the softmax rows of block it+1, then the rest of
//     phi(Q) of block it, its store and the store of P (a bf16 pair hi + lo);
//   K waves (2, 3): phi(K) likewise, stored transposed as hi | lo pairs;
//     with the store, z_{it+1} = z_it + phi(K_it)^T 1 (on the MFMAs, from
//     the tile just stored); with the first half of block it+1, lin_den =
//     phi(Q) z of block it-1 and its merge coefficients;
//   state waves (D/32): the output store of block it-3 (whole rows, from
//     the LDS staging tile the state waves filled an iteration before), the
//     merge of block it-2 (two coefficients per row) into staging; then, for
//     block it-1: the V^T operands of the wave's 32 columns, the readout
//     phi(Q) S against the state of the blocks before it, P V of its
//     columns and the commit into S columns 32w .. 32w+31 (fp32
//     accumulators).
// The QS and K waves hand a block to the state waves through a double
// buffer (written in iteration c, read in c+1), the merge coefficients
// through a second (written in c+1, read in c+2); z goes from one K wave to
// the other through a triple buffer (z_c is written in iteration c-1 and read
// in c and c+1); W_h^T stays in LDS.
// Arithmetic and operand precision are those of the single-group walk above.
// ---------------------------------------------------------------------------
template <typename T, int D, int F>
struct PrefillPipeCfg {
  typedef Mma<T> M;
  typedef typename M::op_t op_t;
  static constexpr int NC = D / kTile;  // state waves
  static constexpr int NWAVE = 4 + NC;
  static constexpr int f = 2 * F;
  static constexpr int NT = F / kTile;
  static constexpr int NPAIR = 2 * NT;
  static constexpr int NRT = f / kTile;
  static constexpr int ZPW = (NRT + NC - 1) / NC;  // z tiles per state wave
  static constexpr int KD = D / M::KW;
  static constexpr int KL = kTile / M::KW;
  static constexpr int KF = f / M::KW;
  // Row strides of the bf16 tiles read as 8-byte pieces by 32 lanes at a
  // time: an odd number of dword pairs, so that the 32 rows fall in distinct
  // bank pairs.
  static constexpr int QLD = f + 4, PLD = kTile + 4;
  struct alignas(16) Buf {            // written in iteration c, read in c + 1
    T phiQ[kTile][QLD];               // phi(q_i)[r] at [i][r]
    uint32_t phiKT[f][kTile + 4];     // phi(k_t)[r] at [r][t]: bf16 hi | lo << 16
    T ph[kTile][PLD];                 // P (relative to the row max) as hi + lo,
    T pl[kTile][PLD];                 //   [query][key]
    float m[kTile], den[kTile];       // row max and sum of the block scores
  };
  struct alignas(16) Smem {
    Buf buf[2];
    float2 coef[2][kTile];            // merge: out = x P V + y phi(Q) S per row
    float z[3][f];                    // z_c at [(c - first block) % 3]
    float stage[2][kTile][D + 4];     // merged outputs of a block, [row][column]
    T vt[NC][kTile][kTile + 8];       // V rows of each state wave's columns
  };
};

template <int D>
constexpr int pipe_threads() {
  return kWave * (4 + D / kTile);
}

template <typename T, int D, int F>
__global__ __launch_bounds__(pipe_threads<D>()) void hyb_prefill_pipe_kernel(
    PrefillArgs a, SegPlan p) {
  typedef PrefillPipeCfg<T, D, F> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  typedef WaveFeatMap<T, D, F> WFM;
  constexpr int f = C::f, E = M::E, KW = M::KW, NT = C::NT, NC = C::NC;
  static_assert(sizeof(T) == 2, "the pipelined walk is the bf16 path");
  static_assert(pipe_threads<D>() == kWave * C::NWAVE, "launch bounds match the waves");
  __shared__ typename C::Smem sh;

  // The wave index through readfirstlane: the compiler then knows it is
  // uniform, and the role branches below are scalar jumps, not exec masks.
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L, T_ = a.T;
  const int units = a.s.B * Hq, nseg = p.nseg, npc = p.npieces();
  const int vix = xcd_unit(blockIdx.x, units * nseg);
  const int u = vix % units, seg = vix / units;
  const int b = u / Hq, h = u % Hq, g = h / (Hq / Hkv);
  const int slot = a.slots ? a.slots[b] : b;
  const bool last = seg == nseg - 1;
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
  const int nblk = T_ / L;
  const int blk0 = seg * p.sb, blk1 = min(nblk, blk0 + p.sb);
  const int nit = blk1 - blk0 + 4;  // iterations blk0-1 .. blk1+2
  if (slot < 0 || slot >= a.s.n_slots) {  // uniform per workgroup
    const size_t ob = ((size_t)b * T_ * Hq + h) * D;
    for (int t = blk0 * L; t < blk1 * L; ++t)
      for (int c = tid; c < D; c += blockDim.x)
        store_out1<T>(a.out, ob + (size_t)t * qstride + c, __builtin_nanf(""), a.s.out_f32);
    return;
  }
  const bool row_ok = li < L;
  const int lrow = min(li, L - 1);
  // Raw buffers over this request's rows of q, k and v: a block's offset is
  // a scalar, a lane's row offset one 32-bit register, a k-step's the
  // immediate (the launcher keeps a request's rows under 2 GiB).
  const __amdgpu_buffer_rsrc_t qrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T*>((const T*)a.q + (size_t)b * T_ * qstride), 0, (int)(T_ * qstride * sizeof(T)),
      kBufferWord3);
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T*>((const T*)a.k + (size_t)b * T_ * kstride), 0, (int)(T_ * kstride * sizeof(T)),
      kBufferWord3);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T*>((const T*)a.v + (size_t)b * T_ * kstride), 0, (int)(T_ * kstride * sizeof(T)),
      kBufferWord3);
  const int qlane = (lrow * (int)qstride + hh * E) * (int)sizeof(T);
  const int klane = (lrow * (int)kstride + hh * E) * (int)sizeof(T);
  auto qoff = [&](int blk) { return (int)(((size_t)blk * L * qstride + (size_t)h * D) * sizeof(T)); };
  auto koff = [&](int blk) { return (int)(((size_t)blk * L * kstride + (size_t)g * D) * sizeof(T)); };
  // Rows of a block tile as operands (rows past the block length read row
  // L-1; the roles mask them).
  auto load_q = [&](int blk, op_t (&o)[C::KD]) {
    const int so = qoff(blk);
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks) o[ks] = buf_op<T>(qrs, qlane + ks * KW * (int)sizeof(T), so);
  };
  auto load_k = [&](int blk, op_t (&o)[C::KD]) {
    const int so = koff(blk);
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks) o[ks] = buf_op<T>(krs, klane + ks * KW * (int)sizeof(T), so);
  };

  // Set-up: z + the earlier segments' increments into z[0].
  {
    const float* __restrict__ wsz = a.ws + (size_t)units * npc * D * f + (size_t)u * npc * f;
    const float* __restrict__ z0 = nseg > 1 ? prefill_snapshot_z(a, npc, u) : a.z + ((size_t)slot * Hq + h) * f;
    for (int r = tid; r < f; r += C::NWAVE * kWave) {
      float zr = z0[r];
      for (int s = 0; s < seg * p.ppseg; ++s) zr += wsz[(size_t)s * f + r];
      sh.z[0][r] = zr;
    }
  }
  lds_barrier();  // z ready

  constexpr float kLog2e = 1.4426950408889634f;
  // logits U^T = W^T X^T of the rows x, from the LDS copy of W_h^T
  // (W_h^T is held in the feature-map waves' registers, wop)
  auto logits = [&](const op_t (&wop)[NT][C::KD], const op_t (&x)[C::KD], float (&phi)[C::NPAIR][16]) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      f32x16 acc = {};
#pragma unroll
      for (int ks = 0; ks < C::KD; ++ks) acc = M::mma(wop[t][ks], x[ks], acc);
#pragma unroll
      for (int i = 0; i < 16; ++i) phi[t][i] = acc[i];
    }
  };
  // Feature-map halves: the row extremes, every first-sign exponential and
  // the first NA of the second sign (the other second-sign slots keep the
  // logit); then the rest, the sums and the normalisation (keep = row_ok
  // zeroes a padding row).  e^(u - mx) = 2^(u log2 e - mx log2 e): one fma
  // per exponent; the rounding of mx log2 e is common to the row and cancels
  // in the ratio.
  auto fm_first = [&](float (&phi)[C::NPAIR][16], int NA, float& mnl, float& sp, float& sn) {
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
    const float mxl = mx * kLog2e;
    mnl = mn * kLog2e;
    sp = 0.0f;
    sn = 0.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float uu = phi[t][i];
        if (t * 16 + i < NA) {
          phi[NT + t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(-uu, kLog2e, mnl));
          sn += phi[NT + t][i];
        } else {
          phi[NT + t][i] = uu;
        }
        phi[t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(uu, kLog2e, -mxl));
        sp += phi[t][i];
      }
  };
  auto fm_second = [&](float (&phi)[C::NPAIR][16], int NA, float mnl, float sp, float sn) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if (t * 16 + i < NA) continue;
        phi[NT + t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(-phi[NT + t][i], kLog2e, mnl));
        sn += phi[NT + t][i];
      }
    sp += xor32(sp);
    sn += xor32(sn);
    const float ip = row_ok ? 1.0f / sp : 0.0f, in = row_ok ? 1.0f / sn : 0.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        phi[t][i] *= ip;
        phi[NT + t][i] *= in;
      }
  };

  if (w < 4) {
    // ---- QS waves (0, 1) and K waves (2, 3): blocks c = blk0 + par + 2j;
    // the first half of block c in iteration c-1, the second in iteration c;
    // the odd wave idles in the first iteration, and both idle after their
    // last block, so that every wave passes nit barriers, as the state waves
    // do ----
    const int par = w & 1;
    op_t ones;
#pragma unroll
    for (int e = 0; e < E; ++e) ones[e] = (T)1.0f;
    auto role = [&](auto key) {
      constexpr bool K = decltype(key)::value;
      // phi(K) stores more (the hi | lo pairs), so it moves more of its
      // exponentials into the first half
      constexpr int NA = K ? NT * 8 : 0;
      op_t x[C::KD], xk[K ? 1 : C::KD], wop[NT][C::KD];
      WFM::load_w((const T*)a.W + (size_t)h * F * D, li, hh, wop);
      auto load = [&](int blk) {
        if constexpr (K) {
          load_k(blk, x);
        } else {
          load_q(blk, x);
          load_k(blk, xk);
        }
      };
      if (blk0 + par < blk1) load(blk0 + par);
      int nbar = 0;
      if (par) {
        lds_barrier();
        ++nbar;
      }
      const float scale = 1.0f / sqrtf((float)D);
      const float lw = log_sigmoid(a.alpha[h]);
      // lin_den = phi(q) . z of block c and the two merge coefficients of
      // each row, for the state waves' merge of block c an iteration later:
      // out = (ca P V + cz phi(Q) S / lin_den) / (ca den + cz), with the
      // overflow-safe ca, cz of the single-group walk; lin_den <= 0 leaves
      // the in-block softmax alone.
      auto coefs = [&](int c) {
        const typename C::Buf& Bc = sh.buf[(c - blk0) & 1];
        const float* zc = sh.z[(c - blk0) % 3];
        float part[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int r = 0; r < f / 2; r += 8) {
          const int r0 = hh * (f / 2) + r;
          const bf16x4 xa = *reinterpret_cast<const bf16x4*>(&Bc.phiQ[li][r0]);
          const bf16x4 xb = *reinterpret_cast<const bf16x4*>(&Bc.phiQ[li][r0 + 4]);
          const f32x4 z0v = *reinterpret_cast<const f32x4*>(zc + r0);
          const f32x4 z1v = *reinterpret_cast<const f32x4*>(zc + r0 + 4);
          const T xt[8] = {xa[0], xa[1], xa[2], xa[3], xb[0], xb[1], xb[2], xb[3]};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            part[e] += to_f32(xt[e]) * z0v[e];
            part[e] += to_f32(xt[4 + e]) * z1v[e];
          }
        }
        float lden = (part[0] + part[1]) + (part[2] + part[3]);
        lden += xor32(lden);
        const float m = Bc.m[li], den = Bc.den[li];
        float ca = 1.0f, cz = 0.0f, rz = 0.0f;
        if (lden > 0.0f) {
          const float la = lw + m, lb = logf(lden);
          const float cc = fmaxf(la, lb);
          ca = expf(la - cc);
          cz = expf(lb - cc);
          rz = 1.0f / lden;
        }
        const float inv = 1.0f / (ca * den + cz);
        if (hh == 0) sh.coef[(c - blk0) & 1][li] = make_float2(ca * inv, cz * rz * inv);
      };
      for (int c = blk0 + par; c < blk1; c += 2) {
        // ---- iteration c-1 ----
        if constexpr (K) {
          if (c - 2 >= blk0) coefs(c - 2);
        }
        float phi[C::NPAIR][16];
        logits(wop, x, phi);
        f32x16 sc = {};
        if constexpr (!K) {
          // scores: keys in rows, queries in columns
#pragma unroll
          for (int ks = 0; ks < C::KD; ++ks)
            sc = M::mma(keep_if<T>(row_ok, xk[ks]), keep_if<T>(row_ok, x[ks]), sc);
        }
        // (the operands are read by the products above before the rows of
        // this wave's next block land in the same registers)
        __builtin_amdgcn_sched_barrier(0);
        if (c + 2 < blk1) load(c + 2);
        float mnl, sp, sn;
        fm_first(phi, NA, mnl, sp, sn);
        float pr[16], m = 0.0f, den = 0.0f;
        if constexpr (!K) {
          m = -INFINITY;
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            pr[i] = row_of(i, hh) < L ? sc[i] * scale : -INFINITY;
            m = fmaxf(m, pr[i]);
          }
          m = fmaxf(m, xor32(m));
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            pr[i] = row_of(i, hh) < L ? fast_exp(pr[i] - m) : 0.0f;
            den += pr[i];
          }
          den += xor32(den);
        }
        lds_barrier();
        // ---- iteration c ----
        fm_second(phi, NA, mnl, sp, sn);
        typename C::Buf& B = sh.buf[(c - blk0) & 1];
        if constexpr (!K) {
#pragma unroll
          for (int p = 0; p < C::NPAIR; ++p)
#pragma unroll
            for (int i = 0; i < 16; ++i) B.phiQ[li][WFM::feature(16 * p + i, hh)] = from_f32<T>(phi[p][i]);
          // P of query li, keys row_of(i, hh): runs of 4 consecutive keys
#pragma unroll
          for (int i = 0; i < 16; i += 4) {
            bf16x4 hi4, lo4;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              hi4[e] = (T)pr[i + e];
              lo4[e] = (T)(pr[i + e] - (float)hi4[e]);
            }
            *reinterpret_cast<bf16x4*>(&B.ph[li][row_of(i, hh)]) = hi4;
            *reinterpret_cast<bf16x4*>(&B.pl[li][row_of(i, hh)]) = lo4;
          }
          if (hh == 0) {
            B.m[li] = m;
            B.den[li] = den;
          }
        } else {
#pragma unroll
          for (int p = 0; p < C::NPAIR; ++p)
#pragma unroll
            for (int i = 0; i < 16; i += 2)
              pack_hi_lo2(phi[p][i], phi[p][i + 1], B.phiKT[WFM::feature(16 * p + i, hh)][li],
                          B.phiKT[WFM::feature(16 * p + i + 1, hh)][li]);
          // z_{c+1} = z_c + phi(K_c)^T 1: the tile just stored read back in
          // operand order (this wave's own LDS writes complete first) as
          // accumulator tiles whose columns are all equal
          asm volatile("" ::: "memory");
          PairRaw kz[C::NRT][C::KL];
#pragma unroll
          for (int p = 0; p < C::NRT; ++p)
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks) kz[p][ks] = lds_pair_raw(&B.phiKT[p * kTile + li][0], ks, hh);
          const float* zc = sh.z[(c - blk0) % 3];
          float* zn = sh.z[(c + 1 - blk0) % 3];
#pragma unroll
          for (int p = 0; p < C::NRT; ++p) {
            f32x16 dz;
#pragma unroll
            for (int i = 0; i < 16; ++i) dz[i] = zc[p * kTile + row_of(i, hh)];
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks) {
              op_t khi, klo;
              pair_split(kz[p][ks], khi, klo);
              dz = M::mma(khi, ones, dz);
              dz = M::mma(klo, ones, dz);
            }
            if (li == 0) {
#pragma unroll
              for (int i = 0; i < 16; i += 4)
                *reinterpret_cast<f32x4*>(&zn[p * kTile + row_of(i, hh)]) =
                    f32x4{dz[i], dz[i + 1], dz[i + 2], dz[i + 3]};
              if (last && c + 1 == blk1) {
                float* zh = a.z + ((size_t)slot * Hq + h) * f;
#pragma unroll
                for (int i = 0; i < 16; i += 4)
                  *reinterpret_cast<f32x4*>(zh + p * kTile + row_of(i, hh)) =
                      f32x4{dz[i], dz[i + 1], dz[i + 2], dz[i + 3]};
              }
            }
          }
        }
        lds_barrier();
        nbar += 2;
      }
      // the coefficients of this wave's last block, an iteration after it
      if constexpr (K) {
        const int clast = blk0 + par + 2 * ((blk1 - blk0 - par - 1) / 2);
        if (clast >= blk0 + par && clast < blk1) {
          coefs(clast);
          lds_barrier();
          ++nbar;
        }
      }
      for (; nbar < nit; ++nbar) lds_barrier();
    };
    if (w >= 2) role(std::true_type{});
    else role(std::false_type{});
  } else {
    // ---- state waves: merge and store of block it-2; V^T, readout, P V
    // and commit of block it-1 ----
    const int cw = w - 4;
    const int col = cw * kTile + li;
    const size_t sbase = (size_t)slot * Hq + h;
    float* __restrict__ Sh = a.S + sbase * f * D;
    const float* __restrict__ wsS = a.ws + (size_t)u * npc * D * f;
    const float* __restrict__ S0 = nseg > 1 ? prefill_snapshot_S(a, npc, u) : Sh;
    // S columns col of all f rows: S + the earlier segments' increments.
    // (Declared here, not before the role branches: a value live across the
    // other roles' code takes registers there too.)
    f32x16 sacc[C::NRT];
#pragma unroll
    for (int rt = 0; rt < C::NRT; ++rt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(S0 + (size_t)col * f + rt * kTile + row_of(4 * j, hh));
#pragma unroll
        for (int r = 0; r < 4; ++r) sacc[rt][4 * j + r] = x[r];
      }
    for (int s = 0; s < seg * p.ppseg; ++s) {
#pragma unroll
      for (int rt = 0; rt < C::NRT; ++rt) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const f32x4 y = *reinterpret_cast<const f32x4*>(
              wsS + (size_t)s * D * f + (size_t)col * f + rt * kTile + row_of(4 * j, hh));
#pragma unroll
          for (int r = 0; r < 4; ++r) sacc[rt][4 * j + r] += y[r];
        }
        // (one row tile of the increment in flight at a time)
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // V rows of this wave's 32 columns, one block ahead: 4 lanes per row
    // (16 bytes each), 16 rows per load; a row at or past the block length
    // reads the next rows of the request (zero past its end) and is zeroed
    // when the operands are formed.  The V^T operands (lane li: column
    // 32cw + li; k-step ks: the tokens row_of(ks*E + e, hh), the order in
    // which P and phi(K)^T enter the products) are then read from this
    // wave's LDS copy of the rows.
    const int vlane = ((lane >> 2) * (int)kstride + cw * kTile + (lane & 3) * 8) * (int)sizeof(T);
    op_t vrow[2];
    auto load_v = [&](int blk) {
      const int so = koff(blk);
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
        vrow[s2] = buf_op<T>(vrs, vlane, so + s2 * 16 * (int)(kstride * sizeof(T)));
    };
    T (*vt)[kTile + 8] = sh.vt[cw];
    if (blk0 < blk1) load_v(blk0);
    // the products of a block, kept from its iteration to its merge in the
    // next
    f32x16 olin = {}, apv = {};
    constexpr int RH = (C::NRT + 1) / 2;
    for (int it = blk0 - 1; it <= blk1 + 2; ++it) {
      const int cr = it - 1, cm = it - 2, cs = it - 3;
      // ---- output store of block cs: this wave's share of the rows of the
      // staging tile, D/8 lanes per row (8 columns, 16 bytes of bf16, each),
      // so that every store covers whole rows ----
      if (cs >= blk0 && cs < blk1) {
        const float (*st)[D + 4] = sh.stage[(cs - blk0) & 1];
        constexpr int LPR = D / 8, RPW = kTile / NC;  // lanes per row, rows per wave
#pragma unroll
        for (int pass = 0; pass < RPW * LPR / kWave; ++pass) {
          const int t = cw * RPW + pass * (kWave / LPR) + lane / LPR, c8 = (lane % LPR) * 8;
          if (t < L) {
            const f32x4 x0 = *reinterpret_cast<const f32x4*>(&st[t][c8]);
            const f32x4 x1 = *reinterpret_cast<const f32x4*>(&st[t][c8 + 4]);
            const float o8[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
            const size_t oidx = (((size_t)b * T_ + (size_t)cs * L + t) * Hq + h) * D + c8;
            store_out8<T>(a.out, oidx, o8, a.s.out_f32);
          }
        }
      }
      // ---- merge of block cm into the staging tile (this wave's columns);
      // stored by all state waves after the next barrier ----
      if (cm >= blk0 && cm < blk1 && row_ok) {
        const float2 cf = sh.coef[(cm - blk0) & 1][li];
        float (*st)[D + 4] = sh.stage[(cm - blk0) & 1];
#pragma unroll
        for (int i = 0; i < 16; i += 4) {
          f32x4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = cf.x * apv[i + e] + cf.y * olin[i + e];
          *reinterpret_cast<f32x4*>(&st[li][cw * kTile + row_of(i, hh)]) = o;
        }
      }
      if (cr >= blk0 && cr < blk1) {
        typename C::Buf& B = sh.buf[(cr - blk0) & 1];
        // LDS operands are requested in batches ahead of the products that
        // use them, a scheduling barrier after each batch: fetched one at a
        // time next to its product, every operand costs a full LDS round
        // trip.  Batch 1: the operands of the readout.
        op_t pb[C::KF];
#pragma unroll
        for (int ks = 0; ks < C::KF; ++ks) pb[ks] = lds_op_perm<T>(&B.phiQ[li][0], ks, hh, 0);
        __builtin_amdgcn_sched_barrier(0);
        // V^T operands of block cr through this wave's LDS rows (its own
        // writes complete before its reads), the next block's rows issued
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
          *reinterpret_cast<op_t*>(&vt[s2 * 16 + (lane >> 2)][(lane & 3) * 8]) = vrow[s2];
        __builtin_amdgcn_sched_barrier(0);
        if (cr + 1 < blk1) load_v(cr + 1);
        asm volatile("" ::: "memory");
        op_t vk[C::KL];
#pragma unroll
        for (int ks = 0; ks < C::KL; ++ks)
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const int t = row_of(ks * E + e, hh);
            vk[ks][e] = t < L ? vt[t][li] : (T)0.0f;
          }
        __builtin_amdgcn_sched_barrier(0);
        // readout against the state of the blocks before cr
        f32x16 ol = {};
#pragma unroll
        for (int ks = 0; ks < C::KF; ++ks) {
          op_t sa;
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const int j = ks * E + e;
            sa[e] = (T)sacc[j / 16][j % 16];
          }
          ol = M::mma(sa, pb[ks], ol);
        }
        __builtin_amdgcn_sched_barrier(0);
        // Batch 2: P of block cr and the commit operands of the first half
        // of the row tiles.
        op_t pph[C::KL], ppl[C::KL];
        PairRaw kr[RH][C::KL];
#pragma unroll
        for (int ks = 0; ks < C::KL; ++ks) {
          pph[ks] = lds_op_perm<T>(&B.ph[li][0], ks, hh, 0);
          ppl[ks] = lds_op_perm<T>(&B.pl[li][0], ks, hh, 0);
        }
#pragma unroll
        for (int rt = 0; rt < RH; ++rt)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) kr[rt][ks] = lds_pair_raw(&B.phiKT[rt * kTile + li][0], ks, hh);
        __builtin_amdgcn_sched_barrier(0);
        // P V of this wave's columns (P as a bf16 pair hi + lo)
        f32x16 pv = {};
#pragma unroll
        for (int ks = 0; ks < C::KL; ++ks) {
          pv = M::mma(vk[ks], pph[ks], pv);
          pv = M::mma(vk[ks], ppl[ks], pv);
        }
        // commit: S += phi(K)^T V (this wave's columns), first half
#pragma unroll
        for (int rt = 0; rt < RH; ++rt)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) {
            op_t khi, klo;
            pair_split(kr[rt][ks], khi, klo);
            sacc[rt] = M::mma(khi, vk[ks], sacc[rt]);
            sacc[rt] = M::mma(klo, vk[ks], sacc[rt]);
          }
        __builtin_amdgcn_sched_barrier(0);
        // Batch 3: the commit operands of the other row tiles.
        PairRaw kr2[C::NRT - RH][C::KL];
#pragma unroll
        for (int rt = RH; rt < C::NRT; ++rt)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks)
            kr2[rt - RH][ks] = lds_pair_raw(&B.phiKT[rt * kTile + li][0], ks, hh);
        __builtin_amdgcn_sched_barrier(0);
        // commit, second half
#pragma unroll
        for (int rt = RH; rt < C::NRT; ++rt)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) {
            op_t khi, klo;
            pair_split(kr2[rt - RH][ks], khi, klo);
            sacc[rt] = M::mma(khi, vk[ks], sacc[rt]);
            sacc[rt] = M::mma(klo, vk[ks], sacc[rt]);
          }
        olin = ol;
        apv = pv;
      }
      lds_barrier();
    }
    if (last) {
#pragma unroll
      for (int rt = 0; rt < C::NRT; ++rt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<f32x4*>(Sh + (size_t)col * f + rt * kTile + row_of(4 * j, hh)) =
              f32x4{sacc[rt][4 * j], sacc[rt][4 * j + 1], sacc[rt][4 * j + 2], sacc[rt][4 * j + 3]};
    }
  }
}


// ---------------------------------------------------------------------------
// Pipelined increment (bf16, F <= 64): the increment of one piece of the
// plan, dS = sum_c phi(K_c)^T V_c and dz = sum_c sum_t phi(k_t), a pair of
// blocks per iteration, 4 + D/32 waves:
//   feature-map waves (4): phi(K) of the piece's blocks, wave w taking the
//     blocks 4m + w; a map spans two iterations (the logits, the row extremes
//     and most exponentials, then the rest and the store of phi(K)^T as
//     hi | lo pairs), so the four waves finish a pair per iteration;
//   state waves (D/32): the commit of the previous pair into S columns
//     32w .. 32w+31 and dz (as phi(K)^T 1) in fp32 accumulators, with the V^T
//     operands of their columns from whole V rows through a per-wave LDS
//     tile.
// One barrier per iteration; phi(K)^T is double-buffered (written in
// iteration j for pair j, read in j + 1).
// ---------------------------------------------------------------------------
template <typename T, int D, int F>
struct DeltaPipeCfg {
  typedef Mma<T> M;
  typedef typename M::op_t op_t;
  static constexpr int NC = D / kTile;   // state waves
  static constexpr int NWAVE = 4 + NC;
  static constexpr int f = 2 * F;
  static constexpr int NT = F / kTile;
  static constexpr int NPAIR = 2 * NT;
  static constexpr int NRT = f / kTile;
  static constexpr int ZPW = (NRT + NC - 1) / NC;  // z tiles per state wave
  static constexpr int KD = D / M::KW;
  static constexpr int KL = kTile / M::KW;
  typedef WaveFeatMap<T, D, F> WFM;
  struct alignas(16) Buf {
    uint32_t phiKT[2][f][kTile + 4];     // per block of the pair: bf16 hi | lo << 16
  };
  struct alignas(16) Smem {
    Buf buf[2];
    T vt[NC][2][kTile][kTile + 8];       // V rows of each state wave's columns
  };
};

template <int D>
constexpr int delta_pipe_threads() {
  return kWave * (4 + D / kTile);
}

template <typename T, int D, int F>
__global__ __launch_bounds__(delta_pipe_threads<D>()) void hyb_prefill_delta_pipe_kernel(
    PrefillArgs a, SegPlan pl) {
  typedef DeltaPipeCfg<T, D, F> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  typedef typename C::WFM WFM;
  constexpr int f = C::f, E = M::E, KW = M::KW, NT = C::NT, NC = C::NC;
  static_assert(sizeof(T) == 2, "the pipelined increment is the bf16 path");
  static_assert(delta_pipe_threads<D>() == kWave * C::NWAVE, "launch bounds match the waves");
  __shared__ typename C::Smem sh;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L, T_ = a.T;
  const int units = a.s.B * Hq;
  // pieces of segments 0 .. nseg-2 (the last segment's increment is never
  // needed)
  const int npc = pl.npieces();
  const int vix = xcd_unit(blockIdx.x, units * npc);
  const int u = vix % units, pc = vix / units;
  const int b = u / Hq, h = u % Hq, g = h / (Hq / Hkv);
  const int slot = a.slots ? a.slots[b] : b;
  if (slot < 0 || slot >= a.s.n_slots) return;  // uniform: no increment needed
  const size_t kstride = (size_t)Hkv * D;
  const int nblk = T_ / L;
  const int blk0 = pl.piece_lo(pc), blk1 = min(nblk, pl.piece_hi(pc));
  const int npair = max(0, (blk1 - blk0 + 1) / 2);
  const int nit = npair + 2;  // iterations -1 .. npair
  const bool row_ok = li < L;
  float* __restrict__ wsS = a.ws + ((size_t)u * npc + pc) * D * f;
  float* __restrict__ wsz = a.ws + (size_t)units * npc * D * f + ((size_t)u * npc + pc) * f;
  // Raw buffers over this request's rows of k and v (the launcher keeps a
  // request's rows under 2 GiB): a block's offset is a scalar.
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T*>((const T*)a.k + (size_t)b * T_ * kstride), 0, (int)(T_ * kstride * sizeof(T)),
      kBufferWord3);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T*>((const T*)a.v + (size_t)b * T_ * kstride), 0, (int)(T_ * kstride * sizeof(T)),
      kBufferWord3);
  auto koff = [&](int blk) { return (int)(((size_t)blk * L * kstride + (size_t)g * D) * sizeof(T)); };
  op_t ones;
#pragma unroll
  for (int e = 0; e < E; ++e) ones[e] = (T)1.0f;

  if (w < 4) {
    // ---- phi(K) of blocks blk0 + w + 4m: the first half in the iteration
    // before the block's pair is due, the second in the pair's iteration;
    // waves 2 and 3 idle in the first iteration, all after their last block,
    // so that every wave passes nit barriers ----
    constexpr float kLog2e = 1.4426950408889634f;
    constexpr int NA = NT * 8;  // second-sign exponentials in the first half
    op_t wop[NT][C::KD], x[C::KD];
    WFM::load_w((const T*)a.W + (size_t)h * F * D, li, hh, wop);
    // rows past the block length read row L-1 (finite); their phi is zeroed
    const int klane = (min(li, L - 1) * (int)kstride + hh * E) * (int)sizeof(T);
    auto load = [&](int blk) {
      const int so = koff(blk);
#pragma unroll
      for (int ks = 0; ks < C::KD; ++ks) x[ks] = buf_op<T>(krs, klane + ks * KW * (int)sizeof(T), so);
    };
    if (blk0 + w < blk1) load(blk0 + w);
    int nbar = 0;
    if (w >> 1) {
      lds_barrier();
      ++nbar;
    }
    for (int c = blk0 + w; c < blk1; c += 4) {
      // ---- first half ----
      float phi[C::NPAIR][16];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        f32x16 acc = {};
#pragma unroll
        for (int ks = 0; ks < C::KD; ++ks) acc = M::mma(wop[t][ks], x[ks], acc);
#pragma unroll
        for (int i = 0; i < 16; ++i) phi[t][i] = acc[i];
      }
      // (the operands are read by the products above before the rows of
      // this wave's next block land in the same registers)
      __builtin_amdgcn_sched_barrier(0);
      if (c + 4 < blk1) load(c + 4);
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
      const float mxl = mx * kLog2e, mnl = mn * kLog2e;
      float sp = 0.0f, sn = 0.0f;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float uu = phi[t][i];
          if (t * 16 + i < NA) {
            phi[NT + t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(-uu, kLog2e, mnl));
            sn += phi[NT + t][i];
          } else {
            phi[NT + t][i] = uu;
          }
          phi[t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(uu, kLog2e, -mxl));
          sp += phi[t][i];
        }
      lds_barrier();
      // ---- second half: the remaining exponentials, the sums,
      // normalisation (keep = row_ok zeroes a padding row) and the store ----
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          if (t * 16 + i < NA) continue;
          phi[NT + t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(-phi[NT + t][i], kLog2e, mnl));
          sn += phi[NT + t][i];
        }
      sp += xor32(sp);
      sn += xor32(sn);
      const float ip = row_ok ? 1.0f / sp : 0.0f, in = row_ok ? 1.0f / sn : 0.0f;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          phi[t][i] *= ip;
          phi[NT + t][i] *= in;
        }
      const int j = (c - blk0) >> 1;
      uint32_t (*kt)[kTile + 4] = sh.buf[j & 1].phiKT[w & 1];
#pragma unroll
      for (int p = 0; p < C::NPAIR; ++p)
#pragma unroll
        for (int i = 0; i < 16; i += 2)
          pack_hi_lo2(phi[p][i], phi[p][i + 1], kt[WFM::feature(16 * p + i, hh)][li],
                      kt[WFM::feature(16 * p + i + 1, hh)][li]);
      lds_barrier();
      nbar += 2;
    }
    for (; nbar < nit; ++nbar) lds_barrier();
  } else {
    // ---- state waves: commit pair i-1 in iteration i ----
    const int cw = w - 4, col = cw * kTile + li;
    f32x16 sacc[C::NRT];
#pragma unroll
    for (int rt = 0; rt < C::NRT; ++rt) sacc[rt] = f32x16{};
    // dz of the feature tiles cw, cw + NC, ... as accumulator tiles whose
    // columns are all equal: phi(K)^T 1 on the MFMAs
    f32x16 zt[C::ZPW];
#pragma unroll
    for (int j = 0; j < C::ZPW; ++j) zt[j] = f32x16{};
    // V rows of this wave's 32 columns for both blocks of a pair, an
    // iteration ahead: 4 lanes per row (16 bytes each), 16 rows per load; a
    // row at or past the block length reads the next rows of the request
    // (zero past its end) and is zeroed when the operands are formed
    const int vlane = ((lane >> 2) * (int)kstride + cw * kTile + (lane & 3) * 8) * (int)sizeof(T);
    op_t vrow[2][2];
    auto load_v = [&](int j) {
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int blk = min(blk0 + 2 * j + q, blk1 - 1);
        const int so = koff(blk);
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
          vrow[q][s2] = buf_op<T>(vrs, vlane, so + s2 * 16 * (int)(kstride * sizeof(T)));
      }
    };
    if (npair > 0) load_v(0);
    op_t ident[C::KL];
#pragma unroll
    for (int ks = 0; ks < C::KL; ++ks)
#pragma unroll
      for (int e = 0; e < E; ++e) ident[ks][e] = (T)(ks * KW + hh * E + e == li ? 1.0f : 0.0f);
    constexpr int RH = (C::NRT + 1) / 2;
    for (int i = -1; i <= npair; ++i) {
      const int j = i - 1;
      if (j >= 0 && j < npair) {
        typename C::Buf& B = sh.buf[j & 1];
        // V^T operands of the pair through this wave's LDS rows (its own
        // writes complete before its reads); the next pair's rows issued
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int s2 = 0; s2 < 2; ++s2)
            *reinterpret_cast<op_t*>(&sh.vt[cw][q][s2 * 16 + (lane >> 2)][(lane & 3) * 8]) = vrow[q][s2];
        __builtin_amdgcn_sched_barrier(0);
        if (j + 1 < npair) load_v(j + 1);
        asm volatile("" ::: "memory");
        // read back as operands (lane li: token li, 16 contiguous bytes of
        // columns per k-step; padding tokens zeroed) and transposed on the
        // MFMAs as V^T = (V I)^T, exact: one nonzero product per entry
        op_t vr[2][C::KL];
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) vr[q][ks] = load_op<T>(&sh.vt[cw][q][li][ks * KW + hh * E]);
        __builtin_amdgcn_sched_barrier(0);
        op_t vk[2][C::KL];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          f32x16 va = {};
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) va = M::mma(keep_if<T>(row_ok, vr[q][ks]), ident[ks], va);
#pragma unroll
          for (int ks = 0; ks < C::KL; ++ks) vk[q][ks] = acc_op_exact<T>(va, ks);
        }
        __builtin_amdgcn_sched_barrier(0);
        // LDS operands in batches ahead of their products (a scheduling
        // barrier after each batch): per block of the pair, the first half
        // of the row tiles, then the rest with z
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          if (blk0 + 2 * j + q >= blk1) continue;  // uniform
          PairRaw kr[RH][C::KL];
#pragma unroll
          for (int rt = 0; rt < RH; ++rt)
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks) kr[rt][ks] = lds_pair_raw(&B.phiKT[q][rt * kTile + li][0], ks, hh);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int rt = 0; rt < RH; ++rt)
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks) {
              op_t khi, klo;
              pair_split(kr[rt][ks], khi, klo);
              sacc[rt] = M::mma(khi, vk[q][ks], sacc[rt]);
              sacc[rt] = M::mma(klo, vk[q][ks], sacc[rt]);
            }
          __builtin_amdgcn_sched_barrier(0);
          PairRaw kr2[C::NRT - RH][C::KL], zr2[C::ZPW][C::KL];
#pragma unroll
          for (int rt = RH; rt < C::NRT; ++rt)
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks)
              kr2[rt - RH][ks] = lds_pair_raw(&B.phiKT[q][rt * kTile + li][0], ks, hh);
#pragma unroll
          for (int jz = 0; jz < C::ZPW; ++jz) {
            const int p = min(cw + jz * NC, C::NRT - 1);
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks) zr2[jz][ks] = lds_pair_raw(&B.phiKT[q][p * kTile + li][0], ks, hh);
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int rt = RH; rt < C::NRT; ++rt)
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks) {
              op_t khi, klo;
              pair_split(kr2[rt - RH][ks], khi, klo);
              sacc[rt] = M::mma(khi, vk[q][ks], sacc[rt]);
              sacc[rt] = M::mma(klo, vk[q][ks], sacc[rt]);
            }
#pragma unroll
          for (int jz = 0; jz < C::ZPW; ++jz) {
            const int p = cw + jz * NC;
            if (p >= C::NRT) continue;  // uniform
#pragma unroll
            for (int ks = 0; ks < C::KL; ++ks) {
              op_t khi, klo;
              pair_split(zr2[jz][ks], khi, klo);
              zt[jz] = M::mma(khi, ones, zt[jz]);
              zt[jz] = M::mma(klo, ones, zt[jz]);
            }
          }
        }
      }
      lds_barrier();
    }
#pragma unroll
    for (int rt = 0; rt < C::NRT; ++rt)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<f32x4*>(wsS + (size_t)col * f + rt * kTile + row_of(4 * j, hh)) =
            f32x4{sacc[rt][4 * j], sacc[rt][4 * j + 1], sacc[rt][4 * j + 2], sacc[rt][4 * j + 3]};
#pragma unroll
    for (int j = 0; j < C::ZPW; ++j) {
      const int p = cw + j * NC;
      if (p < C::NRT && li == 0) {
#pragma unroll
        for (int i = 0; i < 16; i += 4)
          *reinterpret_cast<f32x4*>(wsz + p * kTile + row_of(i, hh)) =
              f32x4{zt[j][i], zt[j][i + 1], zt[j][i + 2], zt[j][i + 3]};
      }
    }
  }
}

template <typename T, int D, int F>
static hipError_t prefill_delta_go(const PrefillArgs& a, const SegPlan& p, hipStream_t st);

template <typename T, int D, int F>
static hipError_t prefill_go(const PrefillArgs& a, hipStream_t st) {
  const int units = a.s.B * a.s.Hq;
  const SegPlan p = prefill_plan(a.s, a.T);
  const dim3 block(kWave * (D / kTile));
  if (p.nseg > 1) {
    // only the last segment walks when no outputs are wanted, and it alone
    // writes the state: no snapshot is needed then
    if (a.out != nullptr) {
      hipLaunchKernelGGL(hyb_prefill_snapshot_kernel, dim3(units), dim3(256), 0, st, a, p.npieces());
      const hipError_t e0 = hipGetLastError();
      if (e0 != hipSuccess) return e0;
    }
    const hipError_t e = prefill_delta_go<T, D, F>(a, p, st);
    if (e != hipSuccess) return e;
  }
  // The pipelined walk serves bf16 with F <= 64 when outputs are wanted;
  // the single-group walk serves the rest.
  if constexpr (sizeof(T) == 2 && F <= 64) {
    // (its buffer loads address a request's rows of q with 32-bit offsets)
    if (a.out != nullptr && (size_t)a.T * a.s.Hq * D * sizeof(T) < ((size_t)1 << 31)) {
      typedef PrefillPipeCfg<T, D, F> P;
      hipLaunchKernelGGL((hyb_prefill_pipe_kernel<T, D, F>), dim3(units * p.nseg),
                         dim3(kWave * P::NWAVE), 0, st, a, p);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((hyb_prefill_kernel<T, D, F>), dim3(units * p.nseg), block, 0, st, a, p, 0);
  return hipGetLastError();
}

template <typename T, int D, int F>
static hipError_t prefill_delta_go(const PrefillArgs& a, const SegPlan& p, hipStream_t st) {
  const int units = a.s.B * a.s.Hq;
  if (p.npieces() <= 0) return hipSuccess;
  if constexpr (sizeof(T) == 2 && F <= 64) {
    hipLaunchKernelGGL((hyb_prefill_delta_pipe_kernel<T, D, F>), dim3(units * p.npieces()),
                       dim3(delta_pipe_threads<D>()), 0, st, a, p);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((hyb_prefill_kernel<T, D, F>), dim3(units * p.npieces()),
                     dim3(kWave * (D / kTile)), 0, st, a, p, 1);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t prefill_delta_f(const PrefillArgs& a, const SegPlan& p, hipStream_t st) {
  switch (a.s.F) {
    case 32: return prefill_delta_go<T, D, 32>(a, p, st);
    case 64: return prefill_delta_go<T, D, 64>(a, p, st);
    case 128: return prefill_delta_go<T, D, 128>(a, p, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_prefill_delta(const PrefillArgs& a, const SegPlan& p, hipStream_t st) {
  if (a.s.dtype == 1)
    return a.s.D == 64 ? prefill_delta_f<bf16, 64>(a, p, st) : prefill_delta_f<bf16, 128>(a, p, st);
  return a.s.D == 64 ? prefill_delta_f<float, 64>(a, p, st) : prefill_delta_f<float, 128>(a, p, st);
}


// The prefill's plan.  A walk workgroup takes a whole CU (its LDS), so the
// walk takes about one workgroup per CU (256 CUs): segments are what the
// batch's (request, head) units leave to fill; at most 8 segments and at
// least 4 blocks per segment.  The increments of segments 0 .. nseg-2 are cut
// into pieces so that they too take about one workgroup per CU, with at
// least 2 blocks per piece (the increment kernel takes blocks in pairs).
SegPlan prefill_plan(const Shape& s, int T) {
  constexpr int kCUs = 256;
  const int units = s.B * s.Hq, nblk = T / s.L;
  int nseg = (kCUs + units - 1) / units;
  if (nseg > 8) nseg = 8;
  if (nseg > nblk / 4) nseg = nblk / 4;
  if (nseg < 1) nseg = 1;
  for (; nseg > 1; --nseg)
    if ((nseg - 1) * ((nblk + nseg - 1) / nseg) < nblk) break;
  SegPlan p;
  p.nseg = nseg;
  p.sb = (nblk + nseg - 1) / nseg;
  p.ppseg = 1;
  p.pb = p.sb;
  if (nseg > 1) {
    int pp = (kCUs + units * (nseg - 1) - 1) / (units * (nseg - 1));
    if (pp > p.sb / 2) pp = p.sb / 2;
    if (pp < 1) pp = 1;
    // every piece non-empty
    for (; pp > 1; --pp)
      if ((pp - 1) * ((p.sb + pp - 1) / pp) < p.sb) break;
    p.ppseg = pp;
    p.pb = (p.sb + pp - 1) / pp;
  }
  return p;
}

// The backward's walks use the prefill's plan: the same one round of walk
// workgroups (a walk workgroup takes a whole CU, and a second round would
// only repeat each workgroup's start, the sum of the earlier increments) and
// the same increment pieces.
SegPlan segment_plan(const Shape& s, int T) { return prefill_plan(s, T); }

size_t prefill_delta_ws_bytes(const Shape& s, const SegPlan& p) {
  if (p.npieces() <= 0) return 0;
  const size_t f = 2 * (size_t)s.F;
  return (size_t)s.B * s.Hq * p.npieces() * ((size_t)s.D * f + f) * 4;
}

size_t prefill_ws_bytes(const Shape& s, int T) {
  const SegPlan p = prefill_plan(s, T);
  if (p.nseg <= 1) return 0;
  const size_t f = 2 * (size_t)s.F;
  // the increments, then the snapshot of the incoming state
  return prefill_delta_ws_bytes(s, p) + (size_t)s.B * s.Hq * ((size_t)s.D * f + f) * 4;
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
