// step.hip -- one denoising step of block-hybrid attention (Section 3.1):
// exact softmax inside the active block, linear readout of the committed
// state, and the gated merge with a shared normaliser.
//
// Decomposition.  One wave per query head and all D output columns: the wave
// computes phi(Q_h), the block softmax and P for its head in registers
// (softmax reductions run over its own accumulators plus two cross-lane
// exchanges), so no work is repeated and heads never wait on each other.  A
// workgroup holds the NW query heads (4 when G = Hq/Hkv allows) that share one
// KV head, and stages that head's V^T through LDS once.  All products use
// 16x16 MFMA tiles, whose operand layout lets four consecutive lanes read 64
// contiguous bytes of a row, so Q, K, W and the state come straight from
// global memory with every 64-byte access fully used.  The state, which
// carries most of the bytes, streams through a double buffer of 16 KiB
// chunks per wave: chunk c+1 is in flight while chunk c is consumed, and the
// first chunk is issued with the block operands at entry.
//
// Every product is computed transposed (columns = queries), so each lane owns
// a query column and the per-query softmax, normaliser and merge are per-lane
// work:
//   Sc^T    = K Q^T / sqrt(D)    -> P^T = exp(Sc^T - max)
//   U^T     = W_h^T Q^T          -> phi(Q)^T
//   lin_den = phi(Q) z
// The merge out = (w sm_num + lin_num) / (w sm_den + lin_den) is folded into
// one accumulator: with per-query coefficients a_q (block branch) and b_q
// (state branch), computed before either product,
//   acc  = V^T (a P)^T            (P carried as bf16 hi + lo)
//   acc += S^T (b phi(Q))^T       (the state streamed in chunks)
// and acc is the output.  With m the block-score maximum, den the max-shifted
// block sum, la = log w + m, lb = log lin_den and c = max(la, lb):
//   a = e^{la-c} / (e^{la-c} den + e^{lb-c}),  b = a e^{lb-la} / lin_den,
// which never overflows; an empty context (lin_den = 0) gives a = 1/den,
// b = 0, plain block softmax.
#include "device.h"
#include "launch.h"

namespace hyb {

template <typename T, int D, int F, int NW>
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
  static constexpr int CB = D / 16;       // 16-column blocks per wave
  static constexpr int CBC = 256 / f;     // column blocks per 64-float state chunk
  static constexpr int NCH = CB / CBC;    // state chunks per wave
  static constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16 bytes
  static constexpr int VT_LD = 36;        // V^T row length (keys, padded)
  static constexpr int NTH = kWave * NW;
  static constexpr int VITEMS = 16 * (D / EPC);    // (key pair, column group)
  static constexpr int VPT = (VITEMS + NTH - 1) / NTH;  // items per thread
  struct alignas(16) Smem {
    T vt[D][VT_LD];   // V^T of the workgroup's KV head, [column][key]
    float z[NW][f];
  };
  static_assert(CBC * NCH == CB, "state chunks must tile the column blocks");

  // Feature held by phi register j (j < NPHI) of a lane in quarter `quad`:
  // j = (sign * FB + fb) * 4 + r -> sign*F + fb*16 + quad*4 + r.
  __device__ static constexpr int feature(int j, int quad) {
    return (j / (4 * FB)) * F + ((j / 4) % FB) * 16 + quad * 4 + (j % 4);
  }
  // Block key held by P register j (j < 8): j = kb*4 + r.
  __device__ static constexpr int key(int j, int quad) {
    return (j / 4) * 16 + quad * 4 + (j % 4);
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

template <typename T, int D, int F, int NW>
__global__ __launch_bounds__(kWave * NW, 1) void hyb_step_kernel(StepArgs a) {
  typedef StepCfg<T, D, F, NW> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  constexpr int f = C::f, E = C::E, KW = C::KW, FB = C::FB, QB = C::QB,
                KB = C::KB, NPHI = C::NPHI, CBC = C::CBC;
  __shared__ typename C::Smem sh;

  const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const int c16 = lane & 15, quad = lane >> 4;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L;
  const int ngrp = Hq / NW;
  const int u = xcd_unit(blockIdx.x, a.s.B * ngrp);
  const int hg = u % ngrp, b = u / ngrp;
  const int h = hg * NW + w, g = (hg * NW) / (Hq / Hkv);
  const int slot = a.slots ? a.slots[b] : b;
  const bool slot_ok = slot >= 0 && slot < a.s.n_slots;
  const size_t sbase = (size_t)(slot_ok ? slot : 0) * Hq + h;
  const float* __restrict__ Sh = a.S + sbase * f * D + c16;
  const float* __restrict__ zh = a.z + sbase * f;
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;
  const T* __restrict__ qb0 = (const T*)a.q + ((size_t)b * L * Hq + h) * D;
  const T* __restrict__ kb0 = (const T*)a.k + ((size_t)b * L * Hkv + g) * D;
  const T* __restrict__ vb0 = (const T*)a.v + ((size_t)b * L * Hkv + g) * D;
  const T* __restrict__ Wt_h = (const T*)a.W + (size_t)h * F * D;

  // 1. Loads, all unconditional and in bounds (rows past the block length
  //    read row L-1 and are masked later).  V and z first: they are staged
  //    into LDS before any math; then Q and K; then the first state chunk.
  uint4 vlo[C::VPT], vhi[C::VPT];  // rows 2kp, 2kp+1 of a 16-byte column group
#pragma unroll
  for (int j = 0; j < C::VPT; ++j) {
    const int it = min(tid + j * C::NTH, C::VITEMS - 1), kp = it % 16, cg = it / 16;
    vlo[j] = *reinterpret_cast<const uint4*>(
        vb0 + (size_t)min(2 * kp, L - 1) * kstride + cg * C::EPC);
    vhi[j] = *reinterpret_cast<const uint4*>(
        vb0 + (size_t)min(2 * kp + 1, L - 1) * kstride + cg * C::EPC);
  }
  constexpr int ZPL = (f + kWave - 1) / kWave;
  float zreg[ZPL];
#pragma unroll
  for (int j = 0; j < ZPL; ++j) zreg[j] = zh[min(lane + j * kWave, f - 1)];
  op_t qop[QB][C::KD], kop[KB][C::KD];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const T* qrow = qb0 + (size_t)min(r * 16 + c16, L - 1) * qstride + quad * E;
    const T* krow = kb0 + (size_t)min(r * 16 + c16, L - 1) * kstride + quad * E;
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks) {
      qop[r][ks] = load_op<T>(qrow + ks * KW);
      kop[r][ks] = load_op<T>(krow + ks * KW);
    }
  }
  // State chunk c: column blocks c*CBC .. c*CBC+CBC-1; element e of k-step
  // ks is state row feature(ks*E + e, quad) -- phi's register order.
  float sch[2][CBC][C::KF][E];
  auto load_chunk = [&](int c) {
#pragma unroll
    for (int cl = 0; cl < CBC; ++cl)
#pragma unroll
      for (int ks = 0; ks < C::KF; ++ks)
#pragma unroll
        for (int e = 0; e < E; ++e)
          sch[c & 1][cl][ks][e] =
              Sh[(size_t)C::feature(ks * E + e, quad) * D + (c * CBC + cl) * 16];
  };
  load_chunk(0);

  // 2. Stage V^T and this head's z, one barrier.
#pragma unroll
  for (int j = 0; j < C::VPT; ++j) {
    const int it = tid + j * C::NTH, kp = it % 16, cg = it / 16;
    if (C::VITEMS % C::NTH != 0 && it >= C::VITEMS) break;
    const T* x0 = reinterpret_cast<const T*>(&vlo[j]);
    const T* x1 = reinterpret_cast<const T*>(&vhi[j]);
#pragma unroll
    for (int e = 0; e < C::EPC; ++e) {
      T* dst = &sh.vt[cg * C::EPC + e][2 * kp];
      dst[0] = 2 * kp < L ? x0[e] : (T)0.0f;
      dst[1] = 2 * kp + 1 < L ? x1[e] : (T)0.0f;
    }
  }
#pragma unroll
  for (int j = 0; j < ZPL; ++j)
    if (lane + j * kWave < f) sh.z[w][lane + j * kWave] = zreg[j];
  __syncthreads();

  // 3. Block scores Sc^T = K Q^T; softmax of query qb*16 + c16 over its 32
  //    keys (8 in this lane, the rest in the other three lane quarters).
  const float scale = 1.0f / sqrtf((float)D);
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
        const bool kv = C::key(kb * 4 + r, quad) < L;
        p[qb][kb * 4 + r] = kv ? sc[r] * scale : -INFINITY;
        m[qb] = fmaxf(m[qb], p[qb][kb * 4 + r]);
      }
    }
    m[qb] = qmax(m[qb]);
    den[qb] = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      p[qb][j] = C::key(j, quad) < L ? fast_exp(p[qb][j] - m[qb]) : 0.0f;
      den[qb] += p[qb][j];
    }
    den[qb] = qsum(den[qb]);
  }

  // 4. U^T = W_h^T Q^T for both query blocks (each W operand loaded once),
  //    then per query block: phi = [softmax(U), softmax(-U)], lin_den =
  //    phi . z, the merge coefficients a (block) and b (state), and b*phi as
  //    the readout's B operand.
  float uu[QB][4 * FB];
#pragma unroll
  for (int fb = 0; fb < FB; ++fb) {
    const T* wrow = Wt_h + (size_t)(fb * 16 + c16) * D + quad * E;
    f32x4 acc[QB] = {};
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks) {
      const op_t wk = load_op<T>(wrow + ks * KW);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) acc[qb] = M::mma(wk, qop[qb][ks], acc[qb]);
    }
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int r = 0; r < 4; ++r) uu[qb][fb * 4 + r] = acc[qb][r];
  }
  const float lw = log_sigmoid(a.alpha[h]);
  op_t phib[QB][C::KF];
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
      phi[j] = fast_exp(uu[qb][j] - mx);
      phi[4 * FB + j] = fast_exp(mn - uu[qb][j]);
      sp += phi[j];
      sn += phi[4 * FB + j];
      zp += phi[j] * sh.z[w][C::feature(j, quad)];
      zn += phi[4 * FB + j] * sh.z[w][C::feature(4 * FB + j, quad)];
    }
    const float ip = 1.0f / qsum(sp), in = 1.0f / qsum(sn);
    const float lden = qsum(zp) * ip + qsum(zn) * in;
    float ca, cb;
    if (lden > 0.0f) {
      const float la = lw + m[qb], lb = logf(lden);
      const float c = fmaxf(la, lb);
      const float ea = expf(la - c), eb = expf(lb - c);
      const float inv = 1.0f / (ea * den[qb] + eb);
      ca = ea * inv;
      cb = eb * inv / lden;
    } else {
      ca = 1.0f / den[qb];
      cb = 0.0f;
    }
    if (!slot_ok) ca = cb = __builtin_nanf("");
#pragma unroll
    for (int j = 0; j < 8; ++j) p[qb][j] *= ca;
    const float sbp = ip * cb, sbn = in * cb;
#pragma unroll
    for (int j = 0; j < NPHI; ++j) phi[j] *= j < 4 * FB ? sbp : sbn;
#pragma unroll
    for (int ks = 0; ks < C::KF; ++ks) phib[qb][ks] = cvt_op<T>(&phi[ks * E]);
  }

  // 5. acc = V^T (aP)^T, then += S^T (b phi)^T chunk by chunk.
  f32x4 acc[C::CB][QB];
#pragma unroll
  for (int cbk = 0; cbk < C::CB; ++cbk)
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      acc[cbk][qb] = f32x4{};
#pragma unroll
      for (int ks = 0; ks < C::KL; ++ks)
        acc[cbk][qb] = mma16_split_b<T>(
            lds_keys_op<T>(&sh.vt[cbk * 16 + c16][0], ks, quad), &p[qb][ks * E],
            acc[cbk][qb]);
    }
#pragma unroll
  for (int c = 0; c < C::NCH; ++c) {
    if (c + 1 < C::NCH) load_chunk(c + 1);
#pragma unroll
    for (int cl = 0; cl < CBC; ++cl)
#pragma unroll
      for (int ks = 0; ks < C::KF; ++ks) {
        const op_t sa = cvt_op<T>(sch[c & 1][cl][ks]);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          acc[c * CBC + cl][qb] = M::mma(sa, phib[qb][ks], acc[c * CBC + cl][qb]);
      }
  }

  // 6. Store: the lane holds query qb*16 + c16, columns cb*16 + quad*4 .. +3.
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    if (qb * 16 + c16 >= L) continue;
    const size_t obase = (((size_t)b * L + qb * 16 + c16) * Hq + h) * D;
#pragma unroll
    for (int cbk = 0; cbk < C::CB; ++cbk) {
      const float o[4] = {acc[cbk][qb][0], acc[cbk][qb][1], acc[cbk][qb][2],
                          acc[cbk][qb][3]};
      store_out4<T>(a.out, obase + cbk * 16 + quad * 4, o, a.s.out_f32);
    }
  }
}

// Heads per workgroup: as many (up to 4) as share one KV head.
static int step_heads_per_wg(int G) {
  return G % 4 == 0 ? 4 : (G % 2 == 0 ? 2 : 1);
}

template <typename T, int D, int F>
static hipError_t step_go(const StepArgs& a, hipStream_t st) {
  const int nw = step_heads_per_wg(a.s.Hq / a.s.Hkv);
  const dim3 grid(a.s.B * (a.s.Hq / nw));
  switch (nw) {
    case 4: hipLaunchKernelGGL((hyb_step_kernel<T, D, F, 4>), grid, dim3(kWave * 4), 0, st, a); break;
    case 2: hipLaunchKernelGGL((hyb_step_kernel<T, D, F, 2>), grid, dim3(kWave * 2), 0, st, a); break;
    default: hipLaunchKernelGGL((hyb_step_kernel<T, D, F, 1>), grid, dim3(kWave), 0, st, a); break;
  }
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t step_f(const StepArgs& a, hipStream_t st) {
  switch (a.s.F) {
    case 32: return step_go<T, D, 32>(a, st);
    case 64: return step_go<T, D, 64>(a, st);
    case 128: return step_go<T, D, 128>(a, st);
  }
  return hipErrorInvalidValue;
}

template <typename T>
static hipError_t step_d(const StepArgs& a, hipStream_t st) {
  switch (a.s.D) {
    case 64: return step_f<T, 64>(a, st);
    case 128: return step_f<T, 128>(a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_step(const StepArgs& a, hipStream_t st) {
  return a.s.dtype == 1 ? step_d<bf16>(a, st) : step_d<float>(a, st);
}

}  // namespace hyb
