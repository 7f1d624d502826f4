// device.h -- gfx950 building blocks shared by the block-hybrid kernels.
//
// Matrix-core conventions.  All products use 32x32 MFMA tiles with fp32
// accumulators:
//   bf16 path:  v_mfma_f32_32x32x16_bf16  (16-deep contraction, 8 bf16/lane)
//   fp32 path:  v_mfma_f32_32x32x2_f32    ( 2-deep contraction, 1 fp32/lane)
// For both, a lane l of the 64-wide wave is split as li = l & 31 and
// hh = l >> 5.  Operand A (M x K) lane (li, hh) holds row li and the E
// contraction indices k = ks*KW + hh*E + e (e < E) of k-step ks; operand B
// (K x N) lane (li, hh) holds column li and the same contraction indices.
// The 16 accumulator registers of lane (li, hh) hold column li and rows
// row_of(i, hh) = (i/4)*8 + hh*4 + i%4, i = 0..15.
//
// Because a contraction does not care in which order its index is visited,
// an accumulator tile can feed the next product directly as an operand:
// register i of lane (li, hh) becomes contraction element e = i % E of
// k-step i / E, provided the other operand is loaded with the same
// (k-step, e, hh) -> index map.  The kernels use this to chain QK^T into
// P V and to read the state straight from its accumulator layout.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hyb {

typedef __bf16 bf16;
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kTile = 32;  // MFMA tile edge, also the largest active block
constexpr int kNumXcd = 8;

template <typename T>
struct Mma;

template <>
struct Mma<bf16> {
  static constexpr int KW = 16;  // contraction depth of one instruction
  static constexpr int E = 8;    // operand elements per lane
  typedef bf16x8 op_t;
  __device__ static inline f32x16 mma(op_t a, op_t b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static inline op_t zero() { return op_t{}; }
};

template <>
struct Mma<float> {
  static constexpr int KW = 2;
  static constexpr int E = 1;
  typedef float op_t;
  __device__ static inline f32x16 mma(op_t a, op_t b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ static inline op_t zero() { return 0.0f; }
};

// 16x16 tiles (gfx950):
//   bf16 path:  v_mfma_f32_16x16x32_bf16  (32-deep contraction, 8 bf16/lane)
//   fp32 path:  v_mfma_f32_16x16x4_f32    ( 4-deep contraction, 1 fp32/lane)
// Lane l is split as c16 = l & 15 and quad = l >> 4.  Operand A (16 x K)
// lane (c16, quad) holds row c16 and contraction indices ks*KW + quad*E + e;
// operand B (K x 16) holds column c16 and the same indices; the 4 accumulator
// registers hold column c16 and rows quad*4 + r.  Four consecutive lanes
// read 64 contiguous bytes of one row, so operands come straight from global
// memory with every 64-byte access fully used.
template <typename T>
struct Mma16;

template <>
struct Mma16<bf16> {
  static constexpr int KW = 32;
  static constexpr int E = 8;
  typedef bf16x8 op_t;
  __device__ static inline f32x4 mma(op_t a, op_t b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static inline op_t zero() { return op_t{}; }
};

template <>
struct Mma16<float> {
  static constexpr int KW = 4;
  static constexpr int E = 1;
  typedef float op_t;
  __device__ static inline f32x4 mma(op_t a, op_t b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  __device__ static inline op_t zero() { return 0.0f; }
};

// The value of lane l ^ 16.  v_permlane16_swap exchanges the odd 16-lane rows
// of its first operand with the even rows of its second: applied to x and x,
// the first result holds rows (0, 0, 2, 2) and the second rows (1, 1, 3, 3),
// so each lane picks the other row of its pair (as xor32 below, no LDS round
// trip).  Blocks are one-dimensional, so bit 4 of the thread index is the
// row's parity.
__device__ inline float xor16(float x) {
  const int v = __builtin_bit_cast(int, x);
  const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return __builtin_bit_cast(float, (threadIdx.x & 16) ? r[0] : r[1]);
}

// Row of accumulator register i (0..15) held by lane half hh.
__device__ __host__ constexpr int row_of(int i, int hh) {
  return (i >> 2) * 8 + hh * 4 + (i & 3);
}

// E consecutive elements of T starting at p (16-byte aligned for bf16).
template <typename T>
__device__ inline typename Mma<T>::op_t load_op(const T* p);
template <>
__device__ inline bf16x8 load_op<bf16>(const bf16* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}
template <>
__device__ inline float load_op<float>(const float* p) {
  return *p;
}

// E consecutive elements of T at byte offset voff + soff of the raw buffer r
// (voff per lane, soff wave-uniform): no 64-bit address per lane.
template <typename T>
__device__ inline typename Mma<T>::op_t buf_op(__amdgpu_buffer_rsrc_t r, int voff, int soff);
template <>
__device__ inline bf16x8 buf_op<bf16>(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
template <>
__device__ inline float buf_op<float>(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

// E fp32 values converted to an operand (bf16 round-to-nearest-even).
template <typename T>
__device__ inline typename Mma<T>::op_t cvt_op(const float* x);
template <>
__device__ inline bf16x8 cvt_op<bf16>(const float* x) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (bf16)x[e];
  return r;
}
template <>
__device__ inline float cvt_op<float>(const float* x) {
  return x[0];
}

// x, or a zero operand when ok is false (a select, not a branch).
// Accumulator registers ks*E .. ks*E+E-1 as a T operand; the tile's rows
// become the contraction index (row_of order).  For values that a T holds
// exactly (a transpose through the identity).
template <typename T>
__device__ inline typename Mma<T>::op_t acc_op_exact(const f32x16& x, int ks) {
  typename Mma<T>::op_t r;
  if constexpr (Mma<T>::E == 1) {
    r = x[ks];
  } else {
#pragma unroll
    for (int e = 0; e < Mma<T>::E; ++e) r[e] = (T)x[ks * Mma<T>::E + e];
  }
  return r;
}

template <typename T>
__device__ inline typename Mma<T>::op_t keep_if(bool ok,
                                               typename Mma<T>::op_t x) {
  return ok ? x : Mma<T>::zero();
}

// Operand whose element e is base[key(e) * stride] for the token
// key(e) = row_of(ks*E + e, hh) (accumulator-row order) or, when natural is
// set, key(e) = ks*KW + hh*E + e; tokens at or beyond L read row L-1 (always
// in bounds) and are replaced by zero.
template <typename T>
__device__ inline typename Mma<T>::op_t load_rows_op(const T* base,
                                                     size_t stride, int ks,
                                                     int hh, int L,
                                                     bool natural) {
  typedef Mma<T> M;
  typename M::op_t x;
  if constexpr (M::E == 1) {
    const int key = natural ? ks * M::KW + hh : row_of(ks, hh);
    const float v = (float)base[(size_t)min(key, L - 1) * stride];
    x = key < L ? v : 0.0f;
  } else {
#pragma unroll
    for (int e = 0; e < M::E; ++e) {
      const int key = natural ? ks * M::KW + hh * M::E + e : row_of(ks * M::E + e, hh);
      const T v = base[(size_t)min(key, L - 1) * stride];
      x[e] = key < L ? v : (T)0.0f;
    }
  }
  return x;
}

// Operand whose element e is row[off + row_of(ks*E + e, hh)]: the LDS copy
// of a tile read in accumulator-register order.  For E = 8 these are two runs
// of 4 consecutive elements.
template <typename T>
__device__ inline typename Mma<T>::op_t lds_op_perm(const T* row, int ks,
                                                    int hh, int off);
template <>
__device__ inline bf16x8 lds_op_perm<bf16>(const bf16* row, int ks, int hh,
                                           int off) {
  const bf16x4 lo = *reinterpret_cast<const bf16x4*>(row + off + 16 * ks + 4 * hh);
  const bf16x4 hi =
      *reinterpret_cast<const bf16x4*>(row + off + 16 * ks + 8 + 4 * hh);
  return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}
template <>
__device__ inline float lds_op_perm<float>(const float* row, int ks, int hh,
                                           int off) {
  return row[off + row_of(ks, hh)];
}

template <typename T>
__device__ inline float to_f32(T x) {
  return (float)x;
}

// The value x takes once it is stored as a T operand (identity for fp32).
template <typename T>
__device__ inline float as_operand(float x) {
  return (float)(T)x;
}

// acc += A * x as T operands, where the E fp32 values x are carried as a
// bf16 pair hi + lo (two products) on the bf16 path: about 16 significant
// bits of x instead of 8.  One product on the fp32 path.
template <typename T>
__device__ inline f32x16 mma_split_b(typename Mma<T>::op_t a, const float* x,
                                     f32x16 acc) {
  typedef Mma<T> M;
  acc = M::mma(a, cvt_op<T>(x), acc);
  if constexpr (M::E > 1) {
    float lo[M::E];
#pragma unroll
    for (int e = 0; e < M::E; ++e) lo[e] = x[e] - as_operand<T>(x[e]);
    acc = M::mma(a, cvt_op<T>(lo), acc);
  }
  return acc;
}

template <typename T>
__device__ inline T from_f32(float x) {
  return (T)x;
}

// Four consecutive outputs at element index idx: fp32 when the call asked
// for fp32 outputs (or computes in fp32), else rounded to T.
template <typename T>
__device__ inline void store_out4(void* out, size_t idx, const float* v,
                                  bool f32) {
  if (sizeof(T) == 4 || f32) {
    *reinterpret_cast<f32x4*>((float*)out + idx) = f32x4{v[0], v[1], v[2], v[3]};
  } else {
    *reinterpret_cast<bf16x4*>((bf16*)out + idx) =
        bf16x4{(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
  }
}

// Eight consecutive outputs at element index idx (16-byte aligned), written
// with non-temporal stores: fp32 as two 16-byte stores, bf16 as one.
template <typename T>
__device__ inline void store_out8_nt(void* out, size_t idx, const float* v,
                                     bool f32) {
  if (sizeof(T) == 4 || f32) {
    f32x4* o = reinterpret_cast<f32x4*>((float*)out + idx);
    __builtin_nontemporal_store(f32x4{v[0], v[1], v[2], v[3]}, o);
    __builtin_nontemporal_store(f32x4{v[4], v[5], v[6], v[7]}, o + 1);
  } else {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const bf16x8 x{(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3],
                   (bf16)v[4], (bf16)v[5], (bf16)v[6], (bf16)v[7]};
    __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(&x),
                                reinterpret_cast<u32x4*>((bf16*)out + idx));
  }
}

// Eight consecutive outputs at element index idx (16-byte aligned): fp32 as
// two 16-byte stores, bf16 as one.
template <typename T>
__device__ inline void store_out8(void* out, size_t idx, const float* v, bool f32) {
  if (sizeof(T) == 4 || f32) {
    f32x4* o = reinterpret_cast<f32x4*>((float*)out + idx);
    o[0] = f32x4{v[0], v[1], v[2], v[3]};
    o[1] = f32x4{v[4], v[5], v[6], v[7]};
  } else {
    *reinterpret_cast<bf16x8*>((bf16*)out + idx) =
        bf16x8{(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3],
               (bf16)v[4], (bf16)v[5], (bf16)v[6], (bf16)v[7]};
  }
}

// x as a bf16 pair in one dword: hi = bf16(x) in the low half, lo =
// bf16(x - hi) in the high half (about 16 significant bits together).
__device__ inline uint32_t pack_hi_lo(float x) {
  const bf16 hi = (bf16)x;
  const bf16 lo = (bf16)(x - (float)hi);
  return (uint32_t)__builtin_bit_cast(uint16_t, hi) |
         ((uint32_t)__builtin_bit_cast(uint16_t, lo) << 16);
}
// pack_hi_lo of two values at once: one paired rounding for the two hi parts
// and one for the two lo parts, then one byte permute per result (the same
// bits as two pack_hi_lo calls).
__device__ inline void pack_hi_lo2(float x0, float x1, uint32_t& p0, uint32_t& p1) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const uint32_t h = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)x0, (__bf16)x1});
  const float h0 = __builtin_bit_cast(float, h << 16);
  const float h1 = __builtin_bit_cast(float, h & 0xffff0000u);
  const uint32_t l = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)(x0 - h0), (__bf16)(x1 - h1)});
  p0 = __builtin_amdgcn_perm(l, h, 0x05040100u);  // h bits 0..15 | l bits 0..15 << 16
  p1 = __builtin_amdgcn_perm(l, h, 0x07060302u);  // h bits 16..31 | l bits 16..31 << 16
}
__device__ inline float unpack_hi(uint32_t p) { return __builtin_bit_cast(float, p << 16); }
__device__ inline float unpack_lo(uint32_t p) { return __builtin_bit_cast(float, p & 0xffff0000u); }

// The hi and lo operands of a row of packed pairs, elements in accumulator
// order (as lds_op_perm): two runs of 4 consecutive entries.  Split into the
// two reads and the unpacking, for callers that request many operands
// before using them.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
struct PairRaw {
  u32x4 a, b;
};
__device__ inline PairRaw lds_pair_raw(const uint32_t* row, int ks, int hh) {
  return PairRaw{*reinterpret_cast<const u32x4*>(row + 16 * ks + 4 * hh),
                 *reinterpret_cast<const u32x4*>(row + 16 * ks + 8 + 4 * hh)};
}
__device__ inline void pair_split(const PairRaw& p, bf16x8& hi, bf16x8& lo) {
  u32x4 h, l;
  // low halves of consecutive dwords -> hi pieces, high halves -> lo pieces
  h[0] = __builtin_amdgcn_perm(p.a[1], p.a[0], 0x05040100u);
  h[1] = __builtin_amdgcn_perm(p.a[3], p.a[2], 0x05040100u);
  h[2] = __builtin_amdgcn_perm(p.b[1], p.b[0], 0x05040100u);
  h[3] = __builtin_amdgcn_perm(p.b[3], p.b[2], 0x05040100u);
  l[0] = __builtin_amdgcn_perm(p.a[1], p.a[0], 0x07060302u);
  l[1] = __builtin_amdgcn_perm(p.a[3], p.a[2], 0x07060302u);
  l[2] = __builtin_amdgcn_perm(p.b[1], p.b[0], 0x07060302u);
  l[3] = __builtin_amdgcn_perm(p.b[3], p.b[2], 0x07060302u);
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}
__device__ inline void lds_pair_op(const uint32_t* row, int ks, int hh, bf16x8& hi,
                                   bf16x8& lo) {
  pair_split(lds_pair_raw(row, ks, hh), hi, lo);
}

// The same for 8 consecutive packed entries (natural order): row + 16*ks +
// 8*hh .. +7.
__device__ inline void lds_pair_op_nat(const uint32_t* row, int ks, int hh, bf16x8& hi,
                                       bf16x8& lo) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 a = *reinterpret_cast<const u32x4*>(row + 16 * ks + 8 * hh);
  const u32x4 b = *reinterpret_cast<const u32x4*>(row + 16 * ks + 8 * hh + 4);
  u32x4 h, l;
  h[0] = __builtin_amdgcn_perm(a[1], a[0], 0x05040100u);
  h[1] = __builtin_amdgcn_perm(a[3], a[2], 0x05040100u);
  h[2] = __builtin_amdgcn_perm(b[1], b[0], 0x05040100u);
  h[3] = __builtin_amdgcn_perm(b[3], b[2], 0x05040100u);
  l[0] = __builtin_amdgcn_perm(a[1], a[0], 0x07060302u);
  l[1] = __builtin_amdgcn_perm(a[3], a[2], 0x07060302u);
  l[2] = __builtin_amdgcn_perm(b[1], b[0], 0x07060302u);
  l[3] = __builtin_amdgcn_perm(b[3], b[2], 0x07060302u);
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}

template <typename T>
__device__ inline void store_out1(void* out, size_t idx, float v, bool f32) {
  if (sizeof(T) == 4 || f32)
    ((float*)out)[idx] = v;
  else
    ((bf16*)out)[idx] = (bf16)v;
}

// The value of lane l ^ 32.  One v_permlane32_swap of x with itself leaves
// the lower half repeated in its first result and the upper half repeated in
// its second, so each lane picks the other half's copy: no LDS round trip
// (as a cross-lane shuffle through ds_bpermute would take).  Waves are 64
// lanes and blocks one-dimensional, so bit 5 of the thread index is the half.
__device__ inline float xor32(float x) {
  const int v = __builtin_bit_cast(int, x);
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __builtin_bit_cast(float, (threadIdx.x & 32) ? r[0] : r[1]);
}

__device__ inline float fast_exp(float x) {
  // e^x = 2^(x log2 e); v_exp_f32 is exact to about 1 ulp.
  return __builtin_amdgcn_exp2f(x * 1.4426950408889634f);
}

constexpr float kLog2e = 1.4426950408889634f;

// 1 / x by the hardware reciprocal (about 1 ulp).
__device__ inline float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// log(sigmoid(a)) without overflow for any a.
__device__ inline float log_sigmoid(float a) {
  return a >= 0.0f ? -log1pf(expf(-a)) : a - log1pf(expf(a));
}

// Workgroup barrier that orders LDS accesses only.  __syncthreads() carries a
// workgroup fence over every address space, which makes each wave wait for
// all of its outstanding global loads before the barrier; restricting the
// fences to the local address space keeps loads issued before the barrier in
// flight (LDS writes are still complete and visible after it).
// Word 3 of a raw buffer resource on gfx9-family chips (32-bit data
// format; the untyped loads and stores used here take no other field).
constexpr int kBufferWord3 = 0x00020000;

// A 16-byte piece per lane from a buffer straight into LDS: lane l's piece
// goes to lds + 16 l (lds is the wave's base, uniform), read from the
// buffer at voff (per lane) + soff (scalar).
__device__ inline void buf_to_lds16(__amdgpu_buffer_rsrc_t r, void* lds, int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff, soff, 0, 0);
}

__device__ inline void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The same ordering for kernels that issue global->LDS copies: the compiler
// counts such a copy as an LDS write until it sees the wave's vmcnt reach 0,
// so before a local fence it waits for every outstanding global load of the
// wave, on whatever path the wave took.  Written out instead: the wave's LDS
// operations complete (lgkmcnt 0), then the barrier; the "memory" clobber
// keeps LDS accesses on their side.  The copies must be waited for
// explicitly (s_waitcnt vmcnt) by the wave that issued them.
__device__ inline void lds_barrier_nodrain() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Work-unit index for the workgroup: consecutive units land on one XCD.
// Workgroups are handed to the 8 XCDs round-robin by blockIdx, so unit
// u = (bid % 8) * (n / 8) + bid / 8 keeps units u..u+n/8-1 on one XCD (and
// in its L2) when n is a multiple of 8.
__device__ inline int xcd_unit(int bid, int n) {
  if ((n & (kNumXcd - 1)) != 0) return bid;
  return (bid & (kNumXcd - 1)) * (n / kNumXcd) + bid / kNumXcd;
}

}  // namespace hyb
