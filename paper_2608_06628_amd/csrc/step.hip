// step.hip -- one denoising step of block-hybrid attention (Section 3.1):
// exact softmax inside the active block, linear readout of the committed
// state, and the gated merge with a shared normaliser.
//
// Decomposition.  A workgroup serves the NW query heads (4 when G = Hq/Hkv
// allows) of one request that share a KV head, with two waves per head:
//
//   block wave  -- Q, K, V, W and z of its head; the block scores and
//                  softmax, phi(Q), lin_den = phi(Q) z, the merge
//                  coefficients, and a P V.  It hands b phi(Q) (as MFMA
//                  operands) and a P V (fp32 accumulators) to the state wave
//                  through LDS, then exits.
//   state wave  -- streams the head's state.  Its first NBUF column blocks
//                  are requested at kernel entry, before anything else.  On
//                  the bf16 path each column block is converted to MFMA
//                  operands as it lands (the fold uses S rounded to bf16
//                  anyway), which frees its buffer for the next request, so
//                  the whole state is requested while the block wave
//                  computes.  After the barrier it folds S^T (b phi)^T onto
//                  a P V column block by column block, the later blocks as
//                  they arrive, and stages the outputs in LDS.
//
// Then all waves write the outputs: a token's NW heads are contiguous in the
// output, so each token is one or two full-wave 16-byte-per-lane stores.
//
// The barriers order LDS only (a workgroup fence restricted to the local
// address space), so the state loads issued before them stay in flight.
//
// Every product is computed transposed (columns = queries), so each lane owns
// one query and the per-query softmax, normaliser and merge are per-lane
// work (16x16 MFMA tiles; lane l = c16 + 16 quad):
//   Sc^T    = K Q^T / sqrt(D)    -> P^T = exp(Sc^T - max)
//   U^T     = W_h^T Q^T          -> phi(Q)^T
//   lin_den = phi(Q) z
// The merge out = (w sm_num + lin_num) / (w sm_den + lin_den) uses per-query
// coefficients a (block branch) and b (state branch):
//   out^T = V^T (a P)^T + S^T (b phi(Q))^T        (P carried as bf16 hi + lo)
// With m the block-score maximum, den the max-shifted block sum,
// la = log w + m, lb = log lin_den and c = max(la, lb):
//   a = e^{la-c} / (e^{la-c} den + e^{lb-c}),  b = a e^{lb-la} / lin_den,
// which never overflows; an empty context (lin_den = 0) gives a = 1/den,
// b = 0, plain block softmax.
//
// State layout: S_h is stored transposed (element (feature r, column c) at
// c*f + r), so the A operand of S^T -- column c16 of a block, four features
// per lane per run -- is one 16-byte load per run.
#include <type_traits>

#include "device.h"
#include "launch.h"

namespace hyb {

// CS > 1 splits each head's output columns (and state columns) over CS
// workgroups: each streams 1/CS of the state and writes 1/CS of the outputs,
// and repeats the per-query block math (small batches, plain step only).
// CO: the commit alone (hybrid_state_commit's grouped kernel): the block
// waves form phi(K) and z, the state waves update S as it lands; no output.
template <typename T, int D, int F, int NW, bool CM = false, int CS = 1, bool CO = false>
struct StepCfg {
  typedef Mma16<T> M;
  typedef typename M::op_t op_t;
  static constexpr int E = M::E, KW = M::KW;
  static constexpr int f = 2 * F;
  static constexpr int FB = F / 16;       // 16-feature blocks per sign
  static constexpr int QB = 2;            // 16-query blocks (32 queries)
  static constexpr int KB = 2;            // 16-key blocks (32 keys)
  static constexpr int NPHI = f / 4;      // phi registers per lane per query block
  static constexpr int KD = D / KW;       // k-steps over head_dim
  static constexpr int KF = f / KW;       // k-steps over features
  static constexpr int KL = 32 / KW;      // k-steps over block keys
  static constexpr int CBF = D / 16;      // 16-column blocks of the output
  static constexpr int CB = CBF / CS;     // ... taken by one workgroup
  static constexpr int RUNS = NPHI / 4;   // 16-byte state runs per column block
  // Column blocks a state wave keeps in flight: 128 registers' worth (192
  // for the commit alone, which holds no readout operands).
  static constexpr int NBUF0 = (CO ? 192 : 128) / (RUNS * 4);
  static constexpr int NBUF = NBUF0 < 1 ? 1 : (NBUF0 > CB ? CB : NBUF0);
  // Column blocks converted to operands before the barrier (bf16 only):
  // enough to have every column block requested, within 64 registers.
  static constexpr int KPK0 = CB - NBUF, KPK1 = 64 / (KF * 4);
  static constexpr int KPACK = (E == 1 || CO) ? 0 : (KPK0 < KPK1 ? KPK0 : KPK1);
  static constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16 bytes
  static constexpr int VT_LD = 36;        // V^T row length (keys, padded)
  static constexpr int VITEMS = 16 * (D / EPC);    // (key pair, column group)
  static constexpr int VPT = (VITEMS + kWave - 1) / kWave;  // items per lane
  // Per head: V^T while the block wave runs, then its a P V accumulators;
  // each pair of column blocks of a P V, once read back, holds the pair's
  // outputs ([32 queries][32 columns], output type).
  union alignas(16) HeadLds {
    T vt[D][VT_LD];
    f32x4 apv[CBF][QB][kWave];
  };
  static_assert(2 * QB * kWave * 16 >= 32 * 32 * 4, "output staging");
  static_assert(CB % 2 == 0, "output columns are stored in pairs of blocks");
  // bf16: the block wave's Q, K, V and (when it fits the head area) W_h rows
  // reach LDS by direct global->LDS copies whose every instruction reads
  // whole rows, 16 bytes per lane; the MFMA operands are then read from LDS,
  // those of V^T by transposing reads.
  static constexpr int CPR = D / EPC;          // 16-byte chunks per row
  static constexpr int RPI = kWave / CPR;      // rows per copy instruction
  static constexpr int RP256 = 256 / (D * (int)sizeof(T)) > 0 ? 256 / (D * (int)sizeof(T)) : 1;
  static constexpr bool DMA_QK = sizeof(T) == 2;
  static constexpr bool DMA_W = DMA_QK && F * D * sizeof(T) <= sizeof(HeadLds);
  // Chunk c of a staged row t sits at position c ^ swz(t), so the 16 rows an
  // operand read takes at one chunk fall in distinct LDS banks.
  __device__ static constexpr int swz(int t) { return (t / RP256) % CPR; }
  // With the commit (CM): phi(K)^T as A operands of phi(K)^T V, per
  // 16-feature block: NPART parts (bf16 hi + lo) x KL key steps.
  static constexpr int NFB = f / 16;
  static constexpr int NPART = E > 1 ? 2 : 1;
  static constexpr int NPK = NPART * KL;
  // Staged Q and K rows are read into registers before b phi(Q) is written
  // over them; the staged V rows are read until the end, so they have their
  // own space.
  struct alignas(16) WaveLds {
    union alignas(16) {
      op_t phib[QB][KF][kWave];  // b phi(Q) as the readout's B operand
      T qk[DMA_QK ? 2 * 32 * D : 1];
    };
    T v[DMA_QK ? 32 * D : 1];
  };
  // Without staged V rows the commit keeps V^T in a space of its own (the
  // head area takes a P V over it).
  static constexpr bool VT_OWN = CM && !DMA_QK;
  // The commit on arrival of the state (bf16, f <= d): the block wave
  // computes phi(K) as soon as its copies land and leaves its operands in
  // consumed staging space -- the bf16 hi parts in the K-staging area (64 d
  // bytes; b phi(Q), 64 f bytes, stays within the Q-staging area before
  // it), the lo parts in the head area (free from the W_h operand reads
  // until a P V) -- so the state wave updates each column block in fp32 as
  // it arrives and never reads the state twice.  Other shapes update in a
  // second pass after the outputs.
  static constexpr bool EARLY = CM && DMA_QK && f <= D;
  static_assert(!EARLY || f * 64 <= (int)sizeof(HeadLds), "phi(K) lo parts in the head area");
  // The grouped commit's staging of an updated column block (16 columns of
  // f floats) in the head area, after the phi(K) lo rows.
  static constexpr int UPD_STG = 32 * D * (int)sizeof(T);
  static_assert(!CO || UPD_STG + 16 * f * 4 <= (int)sizeof(HeadLds), "update staging");
  static_assert(!CO || (f / 4) % 16 == 0, "update staging swizzle");
  // Column blocks held as bf16 readout operands (those converted before b
  // phi(Q) is in LDS; with the early commit the later ones are folded as
  // they arrive).
  static constexpr int NPACK = KPACK;
  // With the early commit, the refill that would request the last column
  // block inside the conversion loop (if one does) waits until b phi(Q) is
  // in LDS and the converted blocks are folded.
  static constexpr bool DEFER = EARLY && CB - 1 - NBUF >= 0 && CB - 1 - NBUF < KPACK;
  struct alignas(16) SmemBase {
    HeadLds hd[NW];  // W_h rows (staged), then V^T, then a P V and outputs
    WaveLds wl[NW];
  };
  struct alignas(16) SmemVt : SmemBase {
    T vt_own[NW][D][VT_LD];
  };
  typedef std::conditional_t<VT_OWN, SmemVt, SmemBase> Smem;
  // Feature held by phi register j (j < NPHI) of a lane in quarter `quad`:
  // j = (sign * FB + fb) * 4 + r -> sign*F + fb*16 + quad*4 + r.
  __device__ static constexpr int feature(int j, int quad) {
    return (j / (4 * FB)) * F + ((j / 4) % FB) * 16 + quad * 4 + (j % 4);
  }
  // Block key held by P register j (j < 8): j = kb*4 + r.
  __device__ static constexpr int key(int j, int quad) {
    return (j / 4) * 16 + quad * 4 + (j % 4);
  }
  // Output column carried by row i of the accumulator tile of column block
  // cb.  Pairs of blocks (2p, 2p+1) cover columns 32p .. 32p+31 so that the
  // lane holding rows quad*4 .. +3 of both blocks owns the 8 consecutive
  // columns 32p + 8 quad .. +7 and stores them with one 16-byte write.
  __device__ static constexpr int column(int cb, int i) {
    return (cb >> 1) * 32 + (i >> 2) * 8 + (cb & 1) * 4 + (i & 3);
  }
};

// Operand whose element e is row[key(ks*E + e, quad)], key as in StepCfg.
template <typename T>
__device__ inline typename Mma16<T>::op_t lds_keys_op(const T* row, int ks,
                                                      int quad);
template <>
__device__ inline bf16x8 lds_keys_op<bf16>(const bf16* row, int ks, int quad) {
  const bf16x4 lo = *reinterpret_cast<const bf16x4*>(row + quad * 4);
  const bf16x4 hi = *reinterpret_cast<const bf16x4*>(row + 16 + quad * 4);
  return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}
template <>
__device__ inline float lds_keys_op<float>(const float* row, int ks, int quad) {
  return row[(ks / 4) * 16 + quad * 4 + (ks % 4)];
}

// acc += A * (x as operand), x carried as a bf16 pair hi + lo on the bf16 path.
template <typename T>
__device__ inline f32x4 mma16_split_b(typename Mma16<T>::op_t a, const float* x,
                                      f32x4 acc) {
  typedef Mma16<T> M;
  acc = M::mma(a, cvt_op<T>(x), acc);
  if constexpr (M::E > 1) {
    float lo[M::E];
#pragma unroll
    for (int e = 0; e < M::E; ++e) lo[e] = x[e] - as_operand<T>(x[e]);
    acc = M::mma(a, cvt_op<T>(lo), acc);
  }
  return acc;
}

// Element e of an MFMA operand set from an fp32 value (rounded to the
// operand type).
template <typename T>
__device__ inline void set_elem(typename Mma16<T>::op_t& o, int e, float x);
template <>
__device__ inline void set_elem<bf16>(bf16x8& o, int e, float x) {
  o[e] = (bf16)x;
}
template <>
__device__ inline void set_elem<float>(float& o, int, float x) {
  o = x;
}

__device__ inline float qmax(float x) {  // max over the 4 lane quarters
  x = fmaxf(x, xor16(x));
  return fmaxf(x, xor32(x));
}
__device__ inline float qmin(float x) {
  x = fminf(x, xor16(x));
  return fminf(x, xor32(x));
}
__device__ inline float qsum(float x) {
  x += xor16(x);
  return x + xor32(x);
}
// max / min / sum over the 16 lanes of a lane quarter (a DPP row, lanes
// c16 = 0..15), on the VALU: swap neighbours, then pairs (quad
// permutations), then combine the two quads of each half-row (half-row
// mirror) and the two halves of the row (row mirror); every lane ends with
// the whole row's result.
template <int CTRL>
__device__ inline float dpp(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
constexpr int kDppSwap1 = 0xB1;       // quad_perm [1, 0, 3, 2]
constexpr int kDppSwap2 = 0x4E;       // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror
constexpr int kDppMirror = 0x140;      // row_mirror
template <typename Op>
__device__ inline float row_reduce16(float x, Op op) {
  x = op(x, dpp<kDppSwap1>(x));
  x = op(x, dpp<kDppSwap2>(x));
  x = op(x, dpp<kDppHalfMirror>(x));
  return op(x, dpp<kDppMirror>(x));
}
__device__ inline float rmax16(float x) {
  return row_reduce16(x, [](float a, float b) { return fmaxf(a, b); });
}
__device__ inline float rmin16(float x) {
  return row_reduce16(x, [](float a, float b) { return fminf(a, b); });
}
__device__ inline float rsum16(float x) {
  return row_reduce16(x, [](float a, float b) { return a + b; });
}

template <typename T, int D, int F, int NW, bool CM, int CS = 1, bool CO = false>
__global__ __launch_bounds__(kWave * 2 * NW, 1) void hyb_step_kernel(StepArgs a) {
  typedef StepCfg<T, D, F, NW, CM, CS, CO> C;
  static_assert(!CO || (CM && C::EARLY), "the commit alone: early-commit shapes only");
  static_assert(CS == 1 || (!CM && sizeof(T) == 2), "column split: plain bf16 step only");
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  constexpr int f = C::f, E = C::E, KW = C::KW, FB = C::FB, QB = C::QB,
                KB = C::KB, NPHI = C::NPHI, RUNS = C::RUNS, NBUF = C::NBUF,
                CB = C::CB;
  __shared__ typename C::Smem sh;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);
  const bool state_wave = wv >= NW;
  const int w = state_wave ? wv - NW : wv;  // head within the group
  const int c16 = lane & 15, quad = lane >> 4;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L;
  const int ngrp = Hq / NW;
  const int uc = xcd_unit(blockIdx.x, a.s.B * ngrp * CS);
  // Column part of a split workgroup: output and state columns coff ..
  // coff + 16 CB - 1.  Pairs of column blocks are whole, so column(cb, i) +
  // coff is the column of local block cb.
  const int coff = (uc % CS) * 16 * C::CB;
  const int u = uc / CS;
  const int hg = u % ngrp, b = u / ngrp;
  const int h = hg * NW + w, g = (hg * NW) / (Hq / Hkv);
  // (uniform through readfirstlane: the state base is then a scalar and
  // each state load needs a 32-bit lane offset, not a 64-bit address)
  const int slot = __builtin_amdgcn_readfirstlane(a.slots ? a.slots[b] : b);
  const bool slot_ok = slot >= 0 && slot < a.s.n_slots;
  // Active tokens of this request's block (the rest are padding: masked as
  // keys, never written as outputs, never committed).
  const int Lb = __builtin_amdgcn_readfirstlane(a.block_len ? min(max(a.block_len[b], 0), L) : L);
  // Rows past Lb read row Lc instead: in bounds, and an active row, so the
  // padding rows are never read whatever they hold.  A request with Lb = 0
  // writes no output and commits nothing.
  const int Lc = max(Lb, 1) - 1;
  const size_t sbase = (size_t)(slot_ok ? slot : 0) * Hq + h;

  // State wave: column block cb of S_h^T; lane (c16, quad) reads the RUNS
  // 16-byte runs of column column(cb, c16) at features feature(4 rn, quad).
  f32x4 buf[NBUF][RUNS];
  const float* __restrict__ St = a.S + sbase * f * D + (size_t)coff * f;
  // Buffer loads over the head's state: the column block's part of the
  // offset is a scalar, the lane's part one VGPR, the run's part the
  // immediate, so a load needs no address arithmetic of its own.
  const __amdgpu_buffer_rsrc_t srs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(St), 0, f * 16 * C::CB * 4, kBufferWord3);
  const int slane = (C::column(0, c16) * f + C::feature(0, quad)) * 4;  // bytes
  auto issue = [&](int cb) {
#pragma unroll
    for (int rn = 0; rn < RUNS; ++rn)
      buf[cb % NBUF][rn] = __builtin_bit_cast(
          f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     srs, slane + (C::feature(rn * 4, 0) - C::feature(0, 0)) * 4,
                     (C::column(cb, 0) - C::column(0, 0)) * f * 4, 0));
  };

  // Staged V rows (bf16) or V^T (fp32) of this head's KV head.
  T* const vst = sh.wl[w].v;
  T(*vt)[C::VT_LD];
  if constexpr (C::VT_OWN)
    vt = sh.vt_own[w];
  else
    vt = sh.hd[w].vt;
  // V^T operands, of a P V and (with the commit) of phi(K)^T V.  The operand
  // of column block cbk holds, in lane (c16, quad), column column(cbk, c16)
  // at keys key(0..7, quad).  From staged V rows: in each 16-lane quarter the
  // transposing read gives lane i element i%4 of the 8-byte pieces addressed
  // by lanes i/4 + 4j (j = 0..3), so lane (i, quad) addresses key
  // quad*4 + i/4 at columns column(cbk, 4*(i%4)) .. +3, four consecutive
  // columns.
  auto vt_op = [&](int cbk, int ks) -> op_t {
    if constexpr (C::DMA_QK) {
      static_assert(C::KL == 1, "one k-step over the block keys");
      typedef short s16x4 __attribute__((ext_vector_type(4)));
      const int col = C::column(cbk, 4 * (c16 % 4)) + coff;
      auto piece = [&](int t) {
        const T* src = vst + t * D + ((col / C::EPC) ^ C::swz(t)) * C::EPC + col % C::EPC;
        return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)src);
      };
      const s16x4 lo = piece(quad * 4 + c16 / 4), hi = piece(16 + quad * 4 + c16 / 4);
      return __builtin_bit_cast(op_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    } else {
      return lds_keys_op<T>(&vt[C::column(cbk, c16) + coff][0], ks, quad);
    }
  };

  // The same transposing reads over rows of another staged tile whose
  // columns are features: lane (c16, quad) gets rows key(0..7, quad) of
  // column col0 + c16 (col0 a multiple of 16), i.e. the phi(K)^T A operand
  // of features col0 .. col0+15 in the key order of vt_op.
  auto rows_op = [&](const T* rows, int col0) -> op_t {
    if constexpr (C::DMA_QK) {
      typedef short s16x4 __attribute__((ext_vector_type(4)));
      const int col = col0 + 4 * (c16 % 4);
      auto piece = [&](int t) {
        const T* src = rows + t * D + ((col / C::EPC) ^ C::swz(t)) * C::EPC + col % C::EPC;
        return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)src);
      };
      const s16x4 lo = piece(quad * 4 + c16 / 4), hi = piece(16 + quad * 4 + c16 / 4);
      return __builtin_bit_cast(op_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    } else {
      return M::zero();
    }
  };

  // K and W_h operands (the block wave's step; the state wave's phi(K) in
  // the commit), z at this lane's features in phi-register order (block
  // wave), phi(K)^T operands (commit, state wave).
  op_t kop[KB][C::KD], wop[FB][C::KD];
  f32x4 zr[RUNS];
  op_t pk[C::NFB][C::NPK];

  // phi(K) of the block keys from kop, wop: U_K = K W_h^T puts feature
  // fb*16 + c16 of keys kb*16 + quad*4 + r in lane (c16, quad), which is the
  // A-operand layout of phi(K)^T V (keys in the order key(j, quad): j =
  // kb*4 + r).  Each key's softmax over the features of a sign reduces
  // across the 16 lanes of its quarter; padding keys get phi = 0.  One
  // 16-key half kb at a time, the four values of 16-feature block fbk go to
  // sink(fbk, part, kb, x4) as part 0 (to be rounded to the operand type)
  // and, when NP = 2, part 1 (the bf16 rounding remainder); zs[fbk] sums the
  // rounded parts over the block keys (feature fbk*16 + c16, every quarter).
  auto phi_k = [&](auto np, float* zs, auto&& sink) {
    constexpr int NP = decltype(np)::value;
#pragma unroll
    for (int fbk = 0; fbk < C::NFB; ++fbk) zs[fbk] = 0.0f;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      float ph[2][FB][4];  // [sign][fb][r]
#pragma unroll
      for (int fb = 0; fb < FB; ++fb) {
        f32x4 acc = {};
#pragma unroll
        for (int ks = 0; ks < C::KD; ++ks) acc = M::mma(kop[kb][ks], wop[fb][ks], acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) ph[0][fb][r] = acc[r];
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float mx = -INFINITY, mn = INFINITY;
#pragma unroll
        for (int fb = 0; fb < FB; ++fb) {
          mx = fmaxf(mx, ph[0][fb][r]);
          mn = fminf(mn, ph[0][fb][r]);
        }
        mx = rmax16(mx);
        mn = rmin16(mn);
        float sp = 0.0f, sn = 0.0f;
#pragma unroll
        for (int fb = 0; fb < FB; ++fb) {
          const float u = ph[0][fb][r];
          ph[0][fb][r] = fast_exp(u - mx);
          ph[1][fb][r] = fast_exp(mn - u);
          sp += ph[0][fb][r];
          sn += ph[1][fb][r];
        }
        // Branch-free: every lane of the row takes part in the reductions.
        const float kv = kb * 16 + quad * 4 + r < Lb ? 1.0f : 0.0f;
        const float ip = kv / rsum16(sp), in = kv / rsum16(sn);
#pragma unroll
        for (int fb = 0; fb < FB; ++fb) {
          ph[0][fb][r] *= ip;
          ph[1][fb][r] *= in;
        }
      }
#pragma unroll
      for (int fbk = 0; fbk < C::NFB; ++fbk) {
        const float* x = ph[fbk / FB][fbk % FB];
        float lo[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          lo[r] = x[r] - as_operand<T>(x[r]);
          zs[fbk] += as_operand<T>(x[r]);
          if constexpr (NP == 2) zs[fbk] += as_operand<T>(lo[r]);
        }
        sink(fbk, 0, kb, x);
        if constexpr (NP == 2) sink(fbk, 1, kb, lo);
      }
    }
#pragma unroll
    for (int fbk = 0; fbk < C::NFB; ++fbk) zs[fbk] = qsum(zs[fbk]);
  };

  // EARLY commit of column block cb (fp32 state in buf): S^T of the block
  // += (phi(K)^T V)^T, the phi(K)^T operands (hi, lo) read by transposing
  // reads from the phi(K) rows the block wave left in its staging space (hi
  // parts over the staged K rows, lo parts in the head area).  Run rn of the
  // block holds, in lane (c16, quad), features rn*16 + quad*4 .. +3 of
  // column column(cb, c16): the accumulator layout of the 16 x 16 tile
  // (features rn*16 .., columns of cb).
  auto update = [&](int cb) {
    if (!slot_ok || Lb == 0) return;
    const T* const pkh = sh.wl[w].qk + 32 * D;
    const T* const pkl = reinterpret_cast<const T*>(&sh.hd[w]);
    const op_t va = vt_op(cb, 0);
    // The updated block goes out through LDS (the second half of the head
    // area, free until a P V): in registers each lane holds 16 bytes of a
    // column, so a direct store would write half-lines; staged as the
    // block's 16 columns of f floats (16-byte chunk k of column i at
    // k ^ (i % 16), conflict-free) it leaves as whole columns, 32 lanes per
    // 512 contiguous bytes.
    // (The commit alone; the fused kernel stores directly: its registers
    // are taken by the readout operands.)
    constexpr int CPC = f / 4;  // 16-byte chunks per column
    f32x4* const stg = reinterpret_cast<f32x4*>(reinterpret_cast<char*>(&sh.hd[w]) + C::UPD_STG);
#pragma unroll
    for (int rn = 0; rn < RUNS; ++rn) {
      f32x4 acc = M::mma(rows_op(pkh, rn * 16), va, buf[cb % NBUF][rn]);
      acc = M::mma(rows_op(pkl, rn * 16), va, acc);
      if constexpr (CO)
        stg[c16 * CPC + ((rn * 4 + quad) ^ c16)] = acc;
      else
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(u32x4, acc), srs, slane + (C::feature(rn * 4, 0) - C::feature(0, 0)) * 4,
            (C::column(cb, 0) - C::column(0, 0)) * f * 4, 0);
    }
    if constexpr (!CO) return;
    // (buffer stores over the head's state: the block's column offset in
    // the scalar offset, the lane's part in one VGPR; one chunk at a time)
    const int rows = kWave / CPC;  // columns per instruction
    const int c0 = lane / CPC, ch = lane % CPC;
#pragma unroll
    for (int j = 0; j < 16 / (kWave / CPC); ++j) {
      const int col = j * rows + c0;
      const f32x4 x = stg[col * CPC + (ch ^ col)];
      __builtin_amdgcn_raw_buffer_store_b128(
          __builtin_bit_cast(u32x4, x), srs,
          ((C::column(0, col) - C::column(0, 0)) * f + ch * 4) * 4,
          (C::column(cb, 0) - C::column(0, 0)) * f * 4, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Column blocks 0 .. KPACK-1 as bf16 operands (S^T A operands).
  op_t sop[C::NPACK > 0 ? C::NPACK : 1][C::KF];
  auto convert = [&](int cb, int ks) {
    float sv[E];
#pragma unroll
    for (int e = 0; e < E; ++e) sv[e] = buf[cb % NBUF][(ks * E + e) / 4][(ks * E + e) % 4];
    return cvt_op<T>(sv);
  };

  const bool of32 = sizeof(T) == 4 || a.s.out_f32;
  // Outputs of the column-block pair pr into the pair's staging area of this
  // head's area: the lane holds query qb*16 + c16 and the 8 consecutive
  // columns 32 pr + 8 quad .. +7 (see column()); acc[0] holds the first
  // block's four, acc[1] the second's.
  auto stage_pair = [&](int pr, const f32x4 (&acc)[2][QB]) {
    char* stg = reinterpret_cast<char*>(&sh.hd[w].apv[2 * pr][0][0]);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const f32x4 lo = acc[0][qb], hi = acc[1][qb];
      const int row = qb * 16 + c16;
      if (of32) {
        f32x4* d = reinterpret_cast<f32x4*>(stg + (row * 32 + quad * 8) * 4);
        d[0] = lo;
        d[1] = hi;
      } else {
        *reinterpret_cast<bf16x8*>(stg + (row * 32 + quad * 8) * 2) =
            bf16x8{(bf16)lo[0], (bf16)lo[1], (bf16)lo[2], (bf16)lo[3],
                   (bf16)hi[0], (bf16)hi[1], (bf16)hi[2], (bf16)hi[3]};
      }
    }
  };

  if (state_wave) {
    if constexpr (C::EARLY) __builtin_amdgcn_s_barrier();  // block requests first
#pragma unroll
    for (int cb = 0; cb < NBUF; ++cb) issue(cb);
    if constexpr (C::EARLY) lds_barrier_nodrain();  // phi(K) is in LDS
#pragma unroll
    for (int cb = 0; cb < C::KPACK; ++cb) {
      if constexpr (C::EARLY) update(cb);
#pragma unroll
      for (int ks = 0; ks < C::KF; ++ks) sop[cb][ks] = convert(cb, ks);
      // Keep the refill below this block's conversion: otherwise the
      // compiler hoists every load to the top and runs out of registers.
#pragma unroll
      for (int ks = 0; ks < C::KF; ++ks) {
        const uint4 t = *reinterpret_cast<const uint4*>(&sop[cb][ks]);
        asm volatile("" ::"v"(t.x), "v"(t.y), "v"(t.z), "v"(t.w) : "memory");
      }
      // (with the early commit the last refill waits for the fold below:
      // its buffer is what the converted blocks need until then)
      if (cb + NBUF < CB && !(C::DEFER && cb + NBUF == CB - 1)) issue(cb + NBUF);
    }
    if constexpr (CO) {
      // The commit alone: each column block is updated as it lands.
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        update(cb);
        if (cb + NBUF < CB) issue(cb + NBUF);
      }
      return;
    } else if constexpr (C::EARLY) {
      // 7. With the early commit the readout folds run inside the update
      //    stream: once b phi(Q) is in LDS, S^T (b phi)^T of the blocks
      //    converted so far, from zero; then each later block is updated,
      //    converted and folded as it arrives.  a P V is added at the end.
      lds_barrier_nodrain();  // b phi(Q) is in LDS
      if constexpr (C::DEFER) issue(CB - 1);
      // (b phi operands are read per column block, not held: the state
      // buffers in flight and the converted blocks fill the registers)
      f32x4 fo[CB][QB];
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        if (cb >= C::KPACK) update(cb);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) fo[cb][qb] = f32x4{};
#pragma unroll
        for (int ks = 0; ks < C::KF; ++ks) {
          const op_t sa = cb < C::KPACK ? sop[cb < C::KPACK ? cb : 0][ks] : convert(cb, ks);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            fo[cb][qb] = M::mma(sa, sh.wl[w].phib[qb][ks][lane], fo[cb][qb]);
        }
        if (cb >= C::KPACK && cb + NBUF < CB) issue(cb + NBUF);
      }
      lds_barrier_nodrain();  // done with phi(K): the head area may take a P V
      lds_barrier_nodrain();  // a P V is in LDS
#pragma unroll
      for (int pr = 0; pr < CB / 2; ++pr) {
        f32x4 acc[2][QB];
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            acc[h2][qb] = sh.hd[w].apv[2 * pr + h2][qb][lane] + fo[2 * pr + h2][qb];
        stage_pair(pr, acc);
      }
      lds_barrier();  // outputs staged
    }
  } else {
    // ---------------- block wave ----------------
    // 1. Loads, all unconditional and in bounds (rows past the request's
    //    block length read row Lc and are masked later).
    const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
    const T* __restrict__ qb0 = (const T*)a.q + ((size_t)b * L * Hq + h) * D;
    const T* __restrict__ kb0 = (const T*)a.k + ((size_t)b * L * Hkv + g) * D;
    const T* __restrict__ vb0 = (const T*)a.v + ((size_t)b * L * Hkv + g) * D;
    const T* __restrict__ Wt_h = (const T*)a.W + (size_t)h * F * D;
    const float* __restrict__ zh = a.z + sbase * f;
    uint4 vlo[C::VPT], vhi[C::VPT];  // rows 2kp, 2kp+1 of a 16-byte column group
    if constexpr (!C::DMA_QK) {
#pragma unroll
      for (int j = 0; j < C::VPT; ++j) {
        const int it = min(lane + j * kWave, C::VITEMS - 1), kp = it % 16, cg = it / 16;
        vlo[j] = *reinterpret_cast<const uint4*>(
            vb0 + (size_t)min(2 * kp, Lc) * kstride + cg * C::EPC);
        vhi[j] = *reinterpret_cast<const uint4*>(
            vb0 + (size_t)min(2 * kp + 1, Lc) * kstride + cg * C::EPC);
      }
    }
    const float alpha_h = CO ? 0.0f : a.alpha[h];
    op_t qop[QB][C::KD];
    T* const wst = reinterpret_cast<T*>(&sh.hd[w]);
    T* const qst = sh.wl[w].qk;
    T* const kst = sh.wl[w].qk + (C::DMA_QK ? 32 * D : 0);
    // Rows 0 .. n-1 of a row-major operand (row t at base + min(t, tmax) *
    // stride) into LDS at dst, chunk-swizzled; copy i takes rows i*RPI ..
    auto stage = [&](const T* base, size_t stride, int n, int tmax, T* dst) {
#pragma unroll
      for (int i = 0; i < n / C::RPI; ++i) {
        const int t = i * C::RPI + lane / C::CPR, pos = lane % C::CPR;
        __builtin_amdgcn_global_load_lds(
            (const __attribute__((address_space(1))) void*)(base + (size_t)min(t, tmax) * stride +
                                                           (pos ^ C::swz(t)) * C::EPC),
            (__attribute__((address_space(3))) void*)(dst + i * C::RPI * D), 16, 0, 0);
      }
    };
    auto staged_op = [&](const T* src, int t, int c) {
      return load_op<T>(src + t * D + (c ^ C::swz(t)) * C::EPC);
    };
    if constexpr (C::DMA_W) stage(Wt_h, D, F, F - 1, wst);
    if constexpr (C::DMA_QK) {
      if constexpr (!CO) stage(qb0, qstride, 32, Lc, qst);
      stage(kb0, kstride, 32, Lc, kst);
      stage(vb0, kstride, 32, Lc, vst);
    } else {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const T* qrow = qb0 + (size_t)min(r * 16 + c16, Lc) * qstride + quad * E;
        const T* krow = kb0 + (size_t)min(r * 16 + c16, Lc) * kstride + quad * E;
#pragma unroll
        for (int ks = 0; ks < C::KD; ++ks) {
          qop[r][ks] = load_op<T>(qrow + ks * KW);
          kop[r][ks] = load_op<T>(krow + ks * KW);
        }
      }
    }
    if constexpr (!C::DMA_W) {
#pragma unroll
      for (int fb = 0; fb < FB; ++fb) {
        const T* wrow = Wt_h + (size_t)(fb * 16 + c16) * D + quad * E;
#pragma unroll
        for (int ks = 0; ks < C::KD; ++ks) wop[fb][ks] = load_op<T>(wrow + ks * KW);
      }
    }
#pragma unroll
    for (int rn = 0; rn < RUNS; ++rn)
      zr[rn] = *reinterpret_cast<const f32x4*>(zh + C::feature(rn * 4, quad));
    // Early commit: the state waves wait for phi(K), which needs these
    // loads first; a plain barrier (no fence, no wait) holds their stream
    // until the block waves' requests are queued ahead of it.
    if constexpr (C::EARLY) __builtin_amdgcn_s_barrier();
    float alpha_v = alpha_h;
    if constexpr (C::DMA_QK) {
      // The copies are counted by vmcnt alone and the compiler does not
      // track them: wait for every load of this wave, then read the operands.
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      // alpha is used only below this wait: without the opaque step the
      // compiler computes log sigmoid(alpha) between the copies and waits
      // there for every copy issued so far (a second memory round trip).
      asm volatile("" : "+v"(alpha_v));
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int ks = 0; ks < C::KD; ++ks) kop[r][ks] = staged_op(kst, r * 16 + c16, quad + 4 * ks);
      if constexpr (C::DMA_W) {
#pragma unroll
        for (int fb = 0; fb < FB; ++fb)
#pragma unroll
          for (int ks = 0; ks < C::KD; ++ks)
            wop[fb][ks] = staged_op(wst, fb * 16 + c16, quad + 4 * ks);
      }
    }
    if constexpr (C::EARLY) {
      // phi(K) for the commit, over the K rows just read (Q is read after
      // it, to keep registers free), one key per lane as phi(Q) below:
      // U_K^T = W_h^T K^T puts features fb*16 + quad*4 + r of key
      // kb*16 + c16 in lane (c16, quad), so each sign's softmax reduces over
      // the four lane quarters; padding keys get phi = 0.  Each key's phi
      // goes to LDS as a row, bf16 hi parts over the staged K rows and lo
      // parts (the rounding remainder) in the head area, chunk-swizzled like
      // the staged V rows; the state wave reads its phi(K)^T operands from
      // them by transposing reads.  z takes the sum of the same rounded
      // values, on the MFMAs (phi(K)^T against a block of ones); z_old is in
      // zr (lane (c16, quad) holds features fbk*16 + quad*4 + r).  Then the
      // state waves may start.
      typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
      T* const pkh = kst;
      T* const pkl = reinterpret_cast<T*>(&sh.hd[w]);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        float u[4 * FB];
#pragma unroll
        for (int fb = 0; fb < FB; ++fb) {
          f32x4 acc = {};
#pragma unroll
          for (int ks = 0; ks < C::KD; ++ks) acc = M::mma(wop[fb][ks], kop[kb][ks], acc);
#pragma unroll
          for (int r = 0; r < 4; ++r) u[fb * 4 + r] = acc[r] * kLog2e;
        }
        float mx = -INFINITY, mn = INFINITY;
#pragma unroll
        for (int j = 0; j < 4 * FB; ++j) {
          mx = fmaxf(mx, u[j]);
          mn = fminf(mn, u[j]);
        }
        mx = qmax(mx);
        mn = qmin(mn);
        float ph[2][4 * FB];
        float sp = 0.0f, sn = 0.0f;
#pragma unroll
        for (int j = 0; j < 4 * FB; ++j) {
          ph[0][j] = __builtin_amdgcn_exp2f(u[j] - mx);
          ph[1][j] = __builtin_amdgcn_exp2f(mn - u[j]);
          sp += ph[0][j];
          sn += ph[1][j];
        }
        const int t = kb * 16 + c16;
        const float kv = t < Lb ? 1.0f : 0.0f;
        const float ip = kv * fast_rcp(qsum(sp)), in = kv * fast_rcp(qsum(sn));
#pragma unroll
        for (int sg = 0; sg < 2; ++sg)
#pragma unroll
          for (int fb = 0; fb < FB; ++fb) {
            const int col = sg * F + fb * 16 + quad * 4;
            const int off = t * D + ((col / C::EPC) ^ C::swz(t)) * C::EPC + col % C::EPC;
            float x[4], lo[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              x[r] = ph[sg][fb * 4 + r] * (sg ? in : ip);
              lo[r] = x[r] - as_operand<T>(x[r]);
            }
            *reinterpret_cast<bf16x4_t*>(pkh + off) = bf16x4_t{(bf16)x[0], (bf16)x[1], (bf16)x[2], (bf16)x[3]};
            *reinterpret_cast<bf16x4_t*>(pkl + off) = bf16x4_t{(bf16)lo[0], (bf16)lo[1], (bf16)lo[2], (bf16)lo[3]};
          }
      }
      asm volatile("" ::: "memory");  // the rows above, then the reads below
      if (slot_ok && Lb > 0) {
        op_t ones;
#pragma unroll
        for (int e = 0; e < E; ++e) set_elem<T>(ones, e, 1.0f);
        float* __restrict__ zw = const_cast<float*>(a.z) + sbase * f;
        // Four feature blocks at a time: every operand read issued before
        // the products, the stores after them.
        constexpr int ZB = C::NFB < 4 ? C::NFB : 4;
        static_assert(C::NFB % ZB == 0, "feature blocks in groups");
#pragma unroll
        for (int f0 = 0; f0 < C::NFB; f0 += ZB) {
          op_t ah[ZB], al[ZB];
#pragma unroll
          for (int i = 0; i < ZB; ++i) {
            ah[i] = rows_op(pkh, (f0 + i) * 16);
            al[i] = rows_op(pkl, (f0 + i) * 16);
          }
          f32x4 zn[ZB];
#pragma unroll
          for (int i = 0; i < ZB; ++i) {
            const f32x4 zs = M::mma(al[i], ones, M::mma(ah[i], ones, f32x4{}));
#pragma unroll
            for (int r = 0; r < 4; ++r) zn[i][r] = zr[f0 + i][r] + zs[r];
          }
          if (c16 == 0) {
#pragma unroll
            for (int i = 0; i < ZB; ++i)
              *reinterpret_cast<f32x4*>(zw + (f0 + i) * 16 + quad * 4) = zn[i];
          }
        }
      }
      lds_barrier_nodrain();
    }
    if constexpr (CO) return;  // the commit alone: phi(K) and z were all
    if constexpr (C::DMA_QK) {
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int ks = 0; ks < C::KD; ++ks) qop[r][ks] = staged_op(qst, r * 16 + c16, quad + 4 * ks);
    }
    // log2 sigmoid(alpha): the merge coefficients are formed in base 2.
    const float lw2 = log_sigmoid(alpha_v) * kLog2e;

    // 2. Without the staged copies: V^T of the KV head into this wave's LDS
    //    area (keys padded to 0).
#pragma unroll
    for (int j = 0; j < (C::DMA_QK ? 0 : C::VPT); ++j) {
      const int it = lane + j * kWave, kp = it % 16, cg = it / 16;
      if (C::VITEMS % kWave != 0 && it >= C::VITEMS) break;
      const T* x0 = reinterpret_cast<const T*>(&vlo[j]);
      const T* x1 = reinterpret_cast<const T*>(&vhi[j]);
#pragma unroll
      for (int e = 0; e < C::EPC; ++e) {
        T* dst = &vt[cg * C::EPC + e][2 * kp];
        dst[0] = 2 * kp < Lb ? x0[e] : (T)0.0f;
        dst[1] = 2 * kp + 1 < Lb ? x1[e] : (T)0.0f;
      }
    }

    // 3. Block scores Sc^T = K Q^T; softmax of query qb*16 + c16 over its 32
    //    keys (8 in this lane, the rest in the other three lane quarters).
    //    Scores are kept in base-2 units (times log2 e), so each weight is
    //    one subtraction and one exp2; m is the maximum in those units.
    const float scale = kLog2e / sqrtf((float)D);
    float p[QB][8], m[QB], den[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      m[qb] = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        f32x4 sc = {};
#pragma unroll
        for (int ks = 0; ks < C::KD; ++ks) sc = M::mma(kop[kb][ks], qop[qb][ks], sc);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool kv = C::key(kb * 4 + r, quad) < Lb;
          p[qb][kb * 4 + r] = kv ? sc[r] * scale : -INFINITY;
          m[qb] = fmaxf(m[qb], p[qb][kb * 4 + r]);
        }
      }
      m[qb] = qmax(m[qb]);
      den[qb] = 0.0f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        p[qb][j] = C::key(j, quad) < Lb ? __builtin_amdgcn_exp2f(p[qb][j] - m[qb]) : 0.0f;
        den[qb] += p[qb][j];
      }
      den[qb] = qsum(den[qb]);
    }

    // 4. U^T = W_h^T Q^T for both query blocks (each W operand used twice).
    float uu[QB][4 * FB];
#pragma unroll
    for (int fb = 0; fb < FB; ++fb) {
      f32x4 acc[QB] = {};
#pragma unroll
      for (int ks = 0; ks < C::KD; ++ks) {
        const op_t wk = wop[fb][ks];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) acc[qb] = M::mma(wk, qop[qb][ks], acc[qb]);
      }
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int r = 0; r < 4; ++r) uu[qb][fb * 4 + r] = acc[qb][r] * kLog2e;
    }

    // 5. Per query block: phi = [softmax(U), softmax(-U)] (U in base-2
    //    units: one subtraction and one exp2 per feature), lin_den = phi z,
    //    the coefficients a and b; a scales P, b phi goes to LDS.
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = -INFINITY, mn = INFINITY;
#pragma unroll
      for (int j = 0; j < 4 * FB; ++j) {
        mx = fmaxf(mx, uu[qb][j]);
        mn = fminf(mn, uu[qb][j]);
      }
      mx = qmax(mx);
      mn = qmin(mn);
      float phi[NPHI];
      float sp = 0.0f, sn = 0.0f, zp = 0.0f, zn = 0.0f;
#pragma unroll
      for (int j = 0; j < 4 * FB; ++j) {
        phi[j] = __builtin_amdgcn_exp2f(uu[qb][j] - mx);
        phi[4 * FB + j] = __builtin_amdgcn_exp2f(mn - uu[qb][j]);
        sp += phi[j];
        sn += phi[4 * FB + j];
        zp += phi[j] * zr[j / 4][j % 4];
        zn += phi[4 * FB + j] * zr[(4 * FB + j) / 4][j % 4];
      }
      const float ip = fast_rcp(qsum(sp)), in = fast_rcp(qsum(sn));
      const float lden = qsum(zp) * ip + qsum(zn) * in;
      // In base 2: la = log2 w + m, lb = log2 lin_den, c = max(la, lb);
      // a = 2^(la-c) / (2^(la-c) den + 2^(lb-c)) and
      // b = 2^(lb-c) / (lin_den (...)) = 2^(-c) / (...).
      float ca, cb;
      if (lden > 0.0f) {
        const float la = lw2 + m[qb], lb = __builtin_amdgcn_logf(lden);
        const float c = fmaxf(la, lb);
        const float ea = __builtin_amdgcn_exp2f(la - c), eb = __builtin_amdgcn_exp2f(lb - c);
        const float inv = fast_rcp(ea * den[qb] + eb);
        ca = ea * inv;
        cb = __builtin_amdgcn_exp2f(-c) * inv;
      } else {
        ca = fast_rcp(den[qb]);
        cb = 0.0f;
      }
      if (!slot_ok) ca = cb = __builtin_nanf("");
#pragma unroll
      for (int j = 0; j < 8; ++j) p[qb][j] *= ca;
      const float sbp = ip * cb, sbn = in * cb;
#pragma unroll
      for (int j = 0; j < NPHI; ++j) phi[j] *= j < 4 * FB ? sbp : sbn;
#pragma unroll
      for (int ks = 0; ks < C::KF; ++ks)
        sh.wl[w].phib[qb][ks][lane] = cvt_op<T>(&phi[ks * E]);
    }
    if constexpr (C::EARLY) lds_barrier_nodrain();  // b phi(Q) is in LDS

    // 6. a P V into accumulators, then over this wave's head area (with
    //    the early commit, once the state wave is done with phi(K): the
    //    products are formed before that barrier, only the stores wait).
    f32x4 acc[CB][QB];
#pragma unroll
    for (int cbk = 0; cbk < CB; ++cbk) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) acc[cbk][qb] = f32x4{};
#pragma unroll
      for (int ks = 0; ks < C::KL; ++ks) {
        const op_t va = vt_op(cbk, ks);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          acc[cbk][qb] = mma16_split_b<T>(va, &p[qb][ks * E], acc[cbk][qb]);
      }
    }
    if constexpr (C::EARLY) lds_barrier_nodrain();
#pragma unroll
    for (int cbk = 0; cbk < CB; ++cbk)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) sh.hd[w].apv[cbk][qb][lane] = acc[cbk][qb];
    if constexpr (C::EARLY) {
      lds_barrier_nodrain();  // a P V is in LDS
      lds_barrier();          // outputs staged
    }
  }
  if constexpr (!C::EARLY) lds_barrier();

  if (!C::EARLY && state_wave) {
    // 7. out^T = a P V + S^T (b phi)^T, a pair of column blocks at a time:
    //    the fold from zero, then a P V added (the arithmetic of the early
    //    commit's fold, so the fused call gives the same bits); column
    //    blocks past KPACK are converted as they land, and each such buffer
    //    is refilled with column block cb + NBUF if not yet requested.
    op_t phib[QB][C::KF];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int ks = 0; ks < C::KF; ++ks) phib[qb][ks] = sh.wl[w].phib[qb][ks][lane];
#pragma unroll
    for (int pr = 0; pr < CB / 2; ++pr) {
      f32x4 acc[2][QB];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int cbk = 2 * pr + h2;
        f32x4 fd[QB] = {};
#pragma unroll
        for (int ks = 0; ks < C::KF; ++ks) {
          const op_t sa = cbk < C::NPACK ? sop[cbk < C::NPACK ? cbk : 0][ks] : convert(cbk, ks);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) fd[qb] = M::mma(sa, phib[qb][ks], fd[qb]);
        }
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) acc[h2][qb] = sh.hd[w].apv[cbk][qb][lane] + fd[qb];
        if (cbk >= C::KPACK && cbk + NBUF < CB) issue(cbk + NBUF);
      }
      // Over the pair's a P V just read.
      stage_pair(pr, acc);
    }
  }
  if constexpr (!C::EARLY) lds_barrier();

  // 8. Store: each wave writes whole tokens (the NW heads of a token are
  //    contiguous, NW * D outputs), 16 bytes per lane; the output is not read
  //    again by this kernel: non-temporal stores.
  {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const int osz = of32 ? 4 : 2;
    const int cph = 16 * C::CB * osz / 16;  // 16-byte chunks per head (this part)
    for (int t = wv; t < Lb; t += 2 * NW) {
      char* orow = reinterpret_cast<char*>(a.out) +
                   ((((size_t)b * L + t) * Hq + hg * NW) * D + coff) * osz;
      for (int c = lane; c < NW * cph; c += kWave) {
        const int hh = c / cph, col0 = (c % cph) * (16 / osz);
        const char* src = reinterpret_cast<const char*>(&sh.hd[hh].apv[2 * (col0 / 32)][0][0]) +
                          (t * 32 + col0 % 32) * osz;
        __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(src),
                                    reinterpret_cast<u32x4*>(orow + (size_t)hh * D * osz +
                                                             (size_t)col0 * osz));
      }
    }
  }

  // 9. With the commit: S_h += phi(K)^T V and z_h += sum_t phi(k_t), by the
  //    state wave once the outputs are out.  It loads K and W_h (from L2),
  //    computes phi(K) of the block keys from U_K = K W_h^T so that lane
  //    (c16, quad) holds feature fb*16 + c16 of keys kb*16 + quad*4 + r:
  //    the A-operand layout of phi(K)^T V (keys in the order key(j, quad)).
  //    Each key's softmax over the features of a sign reduces across the 16
  //    lanes of its quarter; padding keys get phi = 0.  z takes the sum of
  //    the same rounded values that enter S.  Then it reads the state again,
  //    column block by column block, and accumulates onto it in place: run
  //    rn of column block cb holds, in lane (c16, quad), features
  //    rn*16 + quad*4 .. +3 of column column(cb, c16), the accumulator layout
  //    of the 16 x 16 tile (features rn*16 .., columns of cb).  The step above
  //    used the state as it was.
  if constexpr (CM && !C::EARLY) {
    if (state_wave && slot_ok && Lb > 0) {
      static_assert(RUNS == C::NFB, "one state run per 16-feature block");
      {
        const size_t kstride = (size_t)Hkv * D;
        const T* __restrict__ kb0 = (const T*)a.k + ((size_t)b * L * Hkv + g) * D;
        const T* __restrict__ Wt_h = (const T*)a.W + (size_t)h * F * D;
#pragma unroll
        for (int r = 0; r < KB; ++r) {
          const T* krow = kb0 + (size_t)min(r * 16 + c16, Lc) * kstride + quad * E;
#pragma unroll
          for (int ks = 0; ks < C::KD; ++ks) kop[r][ks] = load_op<T>(krow + ks * KW);
        }
#pragma unroll
        for (int fb = 0; fb < FB; ++fb) {
          const T* wrow = Wt_h + (size_t)(fb * 16 + c16) * D + quad * E;
#pragma unroll
          for (int ks = 0; ks < C::KD; ++ks) wop[fb][ks] = load_op<T>(wrow + ks * KW);
        }
      }
      float zs[C::NFB];
      phi_k(std::integral_constant<int, C::NPART>{}, zs, [&](int fbk, int part, int kb, const float* x4) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = kb * 4 + r;  // key(j, quad): operand step j / E, element j % E
          set_elem<T>(pk[fbk][part * C::KL + j / E], j % E, x4[r]);
        }
      });
      // z: lanes c16 == 0 write 16 bytes per 16-feature block.
      {
        float* __restrict__ zw = const_cast<float*>(a.z) + sbase * f;
#pragma unroll
        for (int fbk = 0; fbk < C::NFB; ++fbk) {
          f32x4 zn = *reinterpret_cast<const f32x4*>(zw + fbk * 16 + quad * 4);
#pragma unroll
          for (int r = 0; r < 4; ++r) zn[r] += __shfl(zs[fbk], quad * 4 + r);
          if (c16 == 0) *reinterpret_cast<f32x4*>(zw + fbk * 16 + quad * 4) = zn;
        }
      }
      float* __restrict__ Sw = const_cast<float*>(a.S) + sbase * f * D;
#pragma unroll
      for (int cb = 0; cb < NBUF; ++cb) issue(cb);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        op_t va[C::KL];
#pragma unroll
        for (int ks = 0; ks < C::KL; ++ks) va[ks] = vt_op(cb, ks);
#pragma unroll
        for (int rn = 0; rn < RUNS; ++rn) {
          f32x4 acc = buf[cb % NBUF][rn];
#pragma unroll
          for (int j = 0; j < C::NPK; ++j) acc = M::mma(pk[rn][j], va[j % C::KL], acc);
          *reinterpret_cast<f32x4*>(Sw + (size_t)C::column(cb, c16) * f + C::feature(rn * 4, quad)) =
              acc;
        }
        if (cb + NBUF < CB) issue(cb + NBUF);
      }
    }
  }
}

// Heads per workgroup: as many (up to 4) as share one KV head; fp32 and the
// widest feature map use at most 2, which keeps their two waves per head
// within one SIMD's register file and their LDS within 160 KiB.
template <typename T, int F, bool CM>
constexpr int step_max_heads() {
  return (sizeof(T) == 4 || F == 128) ? 2 : 4;
}

template <typename T, int D, int F, bool CM>
static hipError_t step_go(const StepArgs& a, hipStream_t st) {
  const int G = a.s.Hq / a.s.Hkv;
  int nw = G % 4 == 0 ? 4 : (G % 2 == 0 ? 2 : 1);
  if (nw > step_max_heads<T, F, CM>()) nw = step_max_heads<T, F, CM>();
  const dim3 grid(a.s.B * (a.s.Hq / nw));
  if constexpr (step_max_heads<T, F, CM>() >= 4) {
    static_assert(sizeof(typename StepCfg<T, D, F, 4, CM>::Smem) <= 160 * 1024, "LDS");
    if (nw == 4) {
      hipLaunchKernelGGL((hyb_step_kernel<T, D, F, 4, CM>), grid, dim3(kWave * 8), 0, st, a);
      return hipGetLastError();
    }
  }
  static_assert(sizeof(typename StepCfg<T, D, F, 2, CM>::Smem) <= 160 * 1024, "LDS");
  if (nw == 2)
    hipLaunchKernelGGL((hyb_step_kernel<T, D, F, 2, CM>), grid, dim3(kWave * 4), 0, st, a);
  else
    hipLaunchKernelGGL((hyb_step_kernel<T, D, F, 1, CM>), grid, dim3(kWave * 2), 0, st, a);
  return hipGetLastError();
}

template <typename T, int D, bool CM>
static hipError_t step_f(const StepArgs& a, hipStream_t st) {
  switch (a.s.F) {
    case 32: return step_go<T, D, 32, CM>(a, st);
    case 64: return step_go<T, D, 64, CM>(a, st);
    case 128: return step_go<T, D, 128, CM>(a, st);
  }
  return hipErrorInvalidValue;
}

template <typename T, bool CM>
static hipError_t step_d(const StepArgs& a, hipStream_t st) {
  switch (a.s.D) {
    case 64: return step_f<T, 64, CM>(a, st);
    case 128: return step_f<T, 128, CM>(a, st);
  }
  return hipErrorInvalidValue;
}

// The split kernel while its waves (B Hq d/32, one per unit) fit on the
// chip's 1024 SIMDs at once and the per-head-group grid (B Hq / 4
// workgroups, one per CU) would leave CUs idle.  Measured (16q/4kv, d = 128,
// f = 128, bf16, kernel time): B = 1: 6.1 against 11.1 us; B = 8: 8.4 against
// 12.0; B = 16: 11.7 against 12.6; B = 20 (a second round of waves): 16.8
// against 12.7.
bool step_prefers_split(const Shape& s) {
  return (long)s.B * s.Hq * (s.D / kTile) <= 1024 && (long)s.B * s.Hq / 4 < 256;
}

// The column-split step: bf16, four query heads per workgroup (G a multiple
// of 4, F <= 64, the shapes whose per-head-group kernel takes 4 heads).
bool step_halves_supported(const Shape& s) {
  return s.dtype == 1 && s.F <= 64 && s.Hkv > 0 && (s.Hq / s.Hkv) % 4 == 0;
}

// While the two workgroups per head group fit on the 256 compute units at
// once (the per-head-group grid would leave half of them idle or more).
bool step_prefers_halves(const Shape& s) {
  return step_halves_supported(s) && (long)s.B * (s.Hq / 4) * 2 <= 256;
}

template <int D, int F>
static hipError_t step_halves_go(const StepArgs& a, hipStream_t st) {
  static_assert(sizeof(typename StepCfg<bf16, D, F, 4, false, 2>::Smem) <= 160 * 1024, "LDS");
  const dim3 grid(a.s.B * (a.s.Hq / 4) * 2);
  hipLaunchKernelGGL((hyb_step_kernel<bf16, D, F, 4, false, 2>), grid, dim3(kWave * 8), 0, st, a);
  return hipGetLastError();
}

static hipError_t step_halves(const StepArgs& a, hipStream_t st) {
  if (!step_halves_supported(a.s)) return hipErrorInvalidValue;
  if (a.s.D == 64) return a.s.F == 32 ? step_halves_go<64, 32>(a, st) : step_halves_go<64, 64>(a, st);
  if (a.s.D == 128) return a.s.F == 32 ? step_halves_go<128, 32>(a, st) : step_halves_go<128, 64>(a, st);
  return hipErrorInvalidValue;
}

// Automatic choice: the column split while its workgroups fill at least
// half of the compute units and at most all of them (measured, 16q/4kv,
// d = 128, f = 128, bf16, event-timed calls: B = 12 split 12.1 us against
// halves 12.8; B = 16 split 13.9, halves 12.9; B = 32 whole 18.4, halves
// 14.8), else the split kernel while its waves fit, else one workgroup per
// head group.
hipError_t launch_step(const StepArgs& a, hipStream_t st) {
  int k = a.s.step_kernel;  // 0 auto, 1 split, 2 whole, 3 halves
  if (k == 0) {
    const bool halves = step_prefers_halves(a.s) && (long)a.s.B * (a.s.Hq / 4) * 2 >= 128;
    k = halves ? 3 : step_prefers_split(a.s) ? 1 : step_prefers_halves(a.s) ? 3 : 2;
  }
  if (k == 1) return launch_step_small(a, st);
  if (k == 3) return step_halves(a, st);
  return a.s.dtype == 1 ? step_d<bf16, false>(a, st) : step_d<float, false>(a, st);
}

// hybrid_state_commit with four query heads per workgroup (bf16, f <= d,
// Hq / Hkv a multiple of 4, F <= 64): the fused kernel's early commit
// without the step, so K and V are read once per KV head group, phi(K) is
// formed while the state streams in, and each state column block is
// updated as it lands.
bool commit_grouped_supported(const Shape& s) {
  return s.dtype == 1 && s.F <= 64 && 2 * s.F <= s.D && s.Hkv > 0 && (s.Hq / s.Hkv) % 4 == 0;
}

template <int D, int F>
static hipError_t commit_grouped_go(const StepArgs& a, hipStream_t st) {
  static_assert(sizeof(typename StepCfg<bf16, D, F, 4, true, 1, true>::Smem) <= 160 * 1024, "LDS");
  hipLaunchKernelGGL((hyb_step_kernel<bf16, D, F, 4, true, 1, true>), dim3(a.s.B * (a.s.Hq / 4)),
                     dim3(kWave * 8), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_commit_grouped(const CommitArgs& c, hipStream_t st) {
  if (!commit_grouped_supported(c.s)) return hipErrorInvalidValue;
  StepArgs a{};
  a.s = c.s;
  a.k = c.k;
  a.v = c.v;
  a.W = c.W;
  a.S = c.S;
  a.z = c.z;
  a.slots = c.slots;
  a.block_len = c.block_len;
  if (c.s.D == 128) return c.s.F == 32 ? commit_grouped_go<128, 32>(a, st) : commit_grouped_go<128, 64>(a, st);
  if (c.s.D == 64 && c.s.F == 32) return commit_grouped_go<64, 32>(a, st);
  return hipErrorInvalidValue;
}

// The step of a block's last denoising pass fused with its commit (the
// single launch of Section 3.3): the outputs use the state as it was, then
// S and z take the block's keys and values.  S and z are written in place.
hipError_t launch_step_commit(const StepArgs& a, hipStream_t st) {
  return a.s.dtype == 1 ? step_d<bf16, true>(a, st) : step_d<float, true>(a, st);
}

}  // namespace hyb
