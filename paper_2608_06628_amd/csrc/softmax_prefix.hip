// softmax_prefix.hip -- exact softmax attention of the active block over a
// request's cached prefix plus the block itself: the softmax layer that the
// hybrid layer replaces (Section 2.2 attention without a mask inside the
// block; the comparison of the paper's kernel benchmark, Appendix A).
//
// Split-KV flash decoding.  Keys are indexed in the concatenation
// [k_cache[b][0 .. P_b-1]; k_block[b][0 .. L-1]] and cut into n_split ranges.
// One workgroup per (request b, KV head g, range s) with one wave per query
// head of the group (GQA packing: the G heads share every K/V tile through
// LDS).  Each 32-key tile gives Sc^T = K Q^T (keys in rows, one query per
// lane column), an online-softmax update, and O^T += V^T P^T, with P rounded
// once to the operand type and the running sum taken over the rounded
// weights.  A second kernel merges the ranges with their log-sum-exp weights;
// with a single range the first kernel writes the normalised output itself.
//
// The cache is either contiguous per request ([B][max_prefix][Hkv][d]) or
// paged: a pool of fixed-size pages ([n_pages][page][Hkv][d]) and a page table
// per request, as a serving engine's paged KV cache keeps it (Section 3.3).
// The page size is a power of two of at least 32 rows, so a 32-key tile lies
// in one page.  The ring kernel stages its range's page numbers in LDS when
// it starts (a range holds at most kMaxRange keys), so the copies of a tile
// take their page from LDS and no vector load of the page table sits among
// the copies whose counts the ring waits on.
#include <type_traits>

#include "device.h"
#include "launch.h"

namespace hyb {

template <typename T, int D, int NG>
struct SpCfg {
  typedef Mma<T> M;
  typedef typename M::op_t op_t;
  static constexpr int KD = D / M::KW;
  static constexpr int KL = kTile / M::KW;
  static constexpr int NCT = D / kTile;
  static constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16 bytes
  static constexpr int KLD = D + EPC;              // K rows: 16-byte pad
  static constexpr int VLD = D + 2 * EPC;          // V rows: 32-byte pad
  static constexpr int CPR = D / EPC;              // 16-byte chunks per row
  static constexpr int NCH = (kTile * CPR + kWave * NG - 1) / (kWave * NG);  // per thread
  struct alignas(16) Smem {
    T k[2][kTile][KLD];
    T v[2][kTile][VLD];
  };
};

constexpr int kMaxGroup = 8;  // query heads per KV head handled by one WG
constexpr int kMaxRange = 32768;  // keys of one split range at most
// pages of one range at the smallest page size (32), unaligned ends included
constexpr int kMaxRangePages = kMaxRange / 32 + 2;

// Page of cached token j of a request (page table row ptab), clamped to the
// pool.
__device__ inline int sp_page(const SoftmaxPrefixArgs& a, const int32_t* ptab, int j) {
  const int pg = ptab[j >> a.page_shift];
  return min(max(pg, 0), a.n_pages - 1);
}

// One wave per query head of the KV group; 32-key tiles double-buffered in
// LDS: the tile after next is loaded into registers while the current one is
// computed, and the next one is moved from registers into the free buffer at
// the end of the step, so one barrier per tile orders everything.
template <typename T, int D, int NG, bool PAGED>
__global__ __launch_bounds__(kWave* NG) void hyb_sp_partial_kernel(
    SoftmaxPrefixArgs a, int chunk) {
  typedef SpCfg<T, D, NG> C;
  typedef typename C::M M;
  typedef typename C::op_t op_t;
  constexpr int E = M::E, KW = M::KW, EPC = C::EPC, CPR = C::CPR, NCH = C::NCH;
  __shared__ typename C::Smem sh;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L, G = Hq / Hkv;
  const int ns = a.n_split, Pmax = a.max_prefix;
  const int s = blockIdx.x % ns;
  const int bg = blockIdx.x / ns;
  const int b = bg / Hkv, g = bg % Hkv, h = g * G + w;
  int P = a.prefix_len[b];
  P = P < 0 ? 0 : (P > Pmax ? Pmax : P);
  const int N = P + L;
  const int lo = s * chunk;
  const int hi = min(lo + chunk, N);
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;

  op_t qop[C::KD];
  {
    const T* qrow = (const T*)a.q + ((size_t)b * L * Hq + h) * D +
                    (size_t)li * qstride + hh * E;
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks)
      qop[ks] = li < L ? load_op<T>(qrow + ks * KW) : M::zero();
  }
  // contiguous: this request's rows; paged: the pool, at KV head g
  const T* kc = (const T*)a.k_cache + ((PAGED ? 0 : (size_t)b * Pmax * Hkv) + g) * D;
  const T* vc = (const T*)a.v_cache + ((PAGED ? 0 : (size_t)b * Pmax * Hkv) + g) * D;
  const T* kbk = (const T*)a.k + ((size_t)b * L * Hkv + g) * D;
  const T* vbk = (const T*)a.v + ((size_t)b * L * Hkv + g) * D;
  const int32_t* ptab = PAGED ? a.page_table + (size_t)b * a.max_pages : nullptr;
  // row offset of cached token j (j < P)
  auto crow = [&](int j) __attribute__((always_inline)) -> size_t {
    if constexpr (PAGED)
      return (((size_t)sp_page(a, ptab, j) << a.page_shift) + (j & ((1 << a.page_shift) - 1))) *
             kstride;
    else
      return (size_t)j * kstride;
  };

  // Tile loads: keys past the range read the range's last key (in bounds)
  // and are masked out of the scores below.
  // A tile's share of this thread, held in registers between its load and
  // its move into LDS: nx is the next tile, af the one after it.
  struct TileRegs {
    uint4 k[NCH], v[NCH];
  };
  auto fetch = [&](int j0) __attribute__((always_inline)) {
    TileRegs r;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int idx = tid + c * kWave * NG, key = idx / CPR, part = idx % CPR;
      if (idx < kTile * CPR) {  // (NG not a power of two: a partial last set)
        const int j = min(j0 + key, hi - 1);
        const size_t o = (size_t)part * EPC;
        const size_t cr = j < P ? crow(j) : 0;
        const T* ks = j < P ? kc + cr : kbk + (size_t)(j - P) * kstride;
        const T* vs = j < P ? vc + cr : vbk + (size_t)(j - P) * kstride;
        r.k[c] = *reinterpret_cast<const uint4*>(ks + o);
        r.v[c] = *reinterpret_cast<const uint4*>(vs + o);
      }
    }
    return r;
  };
  auto put = [&](const TileRegs& r, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int idx = tid + c * kWave * NG, key = idx / CPR, part = idx % CPR;
      if (idx < kTile * CPR) {
        *reinterpret_cast<uint4*>(&sh.k[buf][key][part * EPC]) = r.k[c];
        *reinterpret_cast<uint4*>(&sh.v[buf][key][part * EPC]) = r.v[c];
      }
    }
  };
  // V^T operand of column tile ct, k-step ks: lane (li, hh) holds column
  // ct*32 + li at keys row_of(ks*E + e, hh).  bf16: in each 16-lane quarter
  // the transposing read gives lane i element i%4 of the 8-byte pieces
  // addressed by lanes i/4 + 4j (j = 0..3); lane i addresses key
  // kb + i/4 at columns cb + 4*(i%4) .. +3, so it receives keys kb .. kb+3
  // of column cb + i.
  auto vt_op = [&](int buf, int ct, int ks) __attribute__((always_inline)) -> op_t {
    if constexpr (E == 1) {
      return to_f32(sh.v[buf][row_of(ks, hh)][ct * kTile + li]);
    } else {
      typedef short s16x4 __attribute__((ext_vector_type(4)));
      const int i = lane & 15;
      const int cb = ct * kTile + 16 * ((lane >> 4) & 1);
      const int kb = 16 * ks + 4 * hh;
      auto piece = [&](int key) {
        const T* src = &sh.v[buf][key][cb + 4 * (i & 3)];
        return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)src);
      };
      const s16x4 x0 = piece(kb + i / 4), x1 = piece(kb + 8 + i / 4);
      return __builtin_bit_cast(op_t, __builtin_shufflevector(x0, x1, 0, 1, 2, 3, 4, 5, 6, 7));
    }
  };

  const float scale = 1.0f / sqrtf((float)D);
  float m = -INFINITY, l = 0.0f;
  f32x16 acc[C::NCT];
#pragma unroll
  for (int ct = 0; ct < C::NCT; ++ct) acc[ct] = f32x16{};

  TileRegs nx = {}, af = {};
  if (lo < hi) {
    put(fetch(lo), 0);
    if (lo + kTile < hi) nx = fetch(lo + kTile);
  }
  __syncthreads();
  int n = 0;
  for (int j0 = lo; j0 < hi; j0 += kTile, ++n) {
    const int buf = n & 1;
    if (j0 + 2 * kTile < hi) af = fetch(j0 + 2 * kTile);  // tile after next

    f32x16 sc = {};
#pragma unroll
    for (int ks = 0; ks < C::KD; ++ks)
      sc = M::mma(load_op<T>(&sh.k[buf][li][ks * KW + hh * E]), qop[ks], sc);
    // Scaled scores; keys past the range only in the range's last tile
    // (a wave-uniform test, so full tiles carry no masks).
    const bool full = j0 + kTile <= hi;
    float p[16];
    float mt = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      p[i] = (full || j0 + row_of(i, hh) < hi) ? sc[i] * scale : -INFINITY;
      mt = fmaxf(mt, p[i]);
    }
    mt = fmaxf(mt, xor32(mt));
    const float mn = fmaxf(m, mt);
    float ps = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      p[i] = as_operand<T>(fast_exp(p[i] - mn));  // exp(-inf) = 0 past the range
      ps += p[i];
    }
    ps += xor32(ps);
    // The accumulators are rescaled only when some query's running maximum
    // rose: once the maximum settles most tiles skip the 64 multiplies.
    if (__any(mn > m)) {
      const float corr = fast_exp(m - mn);
      l *= corr;
#pragma unroll
      for (int ct = 0; ct < C::NCT; ++ct)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[ct][i] *= corr;
    }
    l += ps;
    m = mn;
#pragma unroll
    for (int ct = 0; ct < C::NCT; ++ct)
#pragma unroll
      for (int ks = 0; ks < C::KL; ++ks)
        acc[ct] = M::mma(vt_op(buf, ct, ks), cvt_op<T>(&p[ks * E]), acc[ct]);
    if (j0 + kTile < hi) put(nx, buf ^ 1);  // next tile into the free buffer
    nx = af;
    __syncthreads();
  }

  // Partial result of this range: unnormalised O, running max and sum.
  if (li >= L) return;
  if (ns == 1) {
    // one range: the result is final, normalised here (no combine launch)
    const float inv = 1.0f / l;
    const size_t ob = (((size_t)b * L + li) * Hq + h) * D;
#pragma unroll
    for (int ct = 0; ct < C::NCT; ++ct)
#pragma unroll
      for (int i = 0; i < 16; i += 4) {
        const float o[4] = {acc[ct][i] * inv, acc[ct][i + 1] * inv, acc[ct][i + 2] * inv,
                            acc[ct][i + 3] * inv};
        store_out4<T>(a.out, ob + ct * kTile + row_of(i, hh), o, a.s.out_f32);
      }
    return;
  }
  const size_t row = (((size_t)b * Hq + h) * ns + s) * L + li;
  float* wacc = (float*)a.ws + row * D;
  float* wml = (float*)a.ws + (size_t)a.s.B * Hq * ns * L * D + row * 2;
#pragma unroll
  for (int ct = 0; ct < C::NCT; ++ct)
#pragma unroll
    for (int i = 0; i < 16; i += 4)
      *reinterpret_cast<f32x4*>(wacc + ct * kTile + row_of(i, hh)) =
          f32x4{acc[ct][i], acc[ct][i + 1], acc[ct][i + 2], acc[ct][i + 3]};
  if (hh == 0) {
    wml[0] = m;
    wml[1] = l;
  }
}


// bf16 with 1, 2, 4 or 8 query heads per KV head: the K/V tiles reach LDS by
// direct global->LDS copies into a ring of R = 4 tile slots, three tiles in
// flight while one is computed, with no registers held for them.  Each copy
// instruction reads whole rows, 16 bytes per lane; chunk c of a staged row t
// sits at position c ^ swz(t), so the rows one operand read touches fall in
// distinct LDS banks.  The slots are distinct arrays and the tile loop is
// unrolled over them, so every copy and every read names its slot at
// compile time.  A wave waits only for its own copies of the tile it is
// about to read (vmcnt counts the later tiles' copies still in flight), then
// one barrier per tile makes all of them visible and frees the slot the
// next copy reuses.
template <int D>
struct SpRing {
  static constexpr int EPC = 8;                      // bf16 per 16 bytes
  static constexpr int CPR = D / EPC;                // chunks per row
  static constexpr int RPI = kWave / CPR;            // rows per copy instruction
  static constexpr int RP256 = 256 / (D * 2) > 0 ? 256 / (D * 2) : 1;
  static constexpr int IK = kTile / RPI;             // copies per 32-row tile
  static constexpr int R = 4;                        // ring slots
  __device__ static constexpr int swz(int t) { return (t / RP256) % CPR; }
};

template <int D>
struct alignas(16) SpSlot {
  bf16 k[kTile * D];
  bf16 v[kTile * D];
};

template <int D, int NG, bool PAGED>
__global__ __launch_bounds__(kWave* NG, 2) void hyb_sp_ring_kernel(SoftmaxPrefixArgs a, int chunk) {
  typedef Mma<bf16> M;
  typedef typename M::op_t op_t;
  typedef SpRing<D> RG;
  constexpr int E = M::E, KW = M::KW, KD = D / KW, KL = kTile / KW, NCT = D / kTile;
  constexpr int EPC = RG::EPC, CPR = RG::CPR, RPI = RG::RPI, IK = RG::IK, R = RG::R;
  constexpr int IPW = 2 * IK / NG;  // copies per wave per tile
  static_assert(IPW * NG == 2 * IK, "copies split evenly over the waves");
  __shared__ SpSlot<D> s0, s1, s2, s3;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int li = lane & 31, hh = lane >> 5;
  const int Hq = a.s.Hq, Hkv = a.s.Hkv, L = a.s.L, G = Hq / Hkv;
  const int ns = a.n_split, Pmax = a.max_prefix;
  // The KV head varies fastest: the Hkv workgroups that read the same
  // token rows of the cache (each its 1/Hkv share of every row) start
  // together.
  const int g = blockIdx.x % Hkv;
  const int s = (blockIdx.x / Hkv) % ns;
  const int b = blockIdx.x / (Hkv * ns), h = g * G + w;
  int P = a.prefix_len[b];
  P = P < 0 ? 0 : (P > Pmax ? Pmax : P);
  const int N = P + L;
  const int lo = s * chunk;
  const int hi = min(lo + chunk, N);
  const int ntiles = hi > lo ? (hi - lo + kTile - 1) / kTile : 0;
  const size_t qstride = (size_t)Hq * D, kstride = (size_t)Hkv * D;

  op_t qop[KD];
  {
    const bf16* qrow = (const bf16*)a.q + ((size_t)b * L * Hq + h) * D + (size_t)li * qstride + hh * E;
#pragma unroll
    for (int ks = 0; ks < KD; ++ks) qop[ks] = li < L ? load_op<bf16>(qrow + ks * KW) : M::zero();
  }
  // contiguous: this request's rows; paged: the pool, at KV head g
  const bf16* kc = (const bf16*)a.k_cache + ((PAGED ? 0 : (size_t)b * Pmax * Hkv) + g) * D;
  const bf16* vc = (const bf16*)a.v_cache + ((PAGED ? 0 : (size_t)b * Pmax * Hkv) + g) * D;
  const bf16* kbk = (const bf16*)a.k + ((size_t)b * L * Hkv + g) * D;
  const bf16* vbk = (const bf16*)a.v + ((size_t)b * L * Hkv + g) * D;
  // Paged: the pages of the cached keys of this range, lo .. min(hi, P) - 1,
  // staged in LDS (page index p0 + e at e), clamped to the pool.
  __shared__ int pages[PAGED ? kMaxRangePages : 1];
  const int p0 = lo >> a.page_shift;
  if constexpr (PAGED) {
    const int32_t* ptab = a.page_table + (size_t)b * a.max_pages;
    const int chi = min(hi, P);
    const int np = chi > lo ? ((chi - 1) >> a.page_shift) - p0 + 1 : 0;
    for (int e = tid; e < np; e += kWave * NG) pages[e] = sp_page(a, ptab, (p0 + e) << a.page_shift);
    __syncthreads();
  }

  // Copies of a tile that lies wholly in the cached prefix: a buffer
  // descriptor whose base is the tile's first row (a scalar) and, per lane
  // and copy, the 32-bit offset of its 16-byte piece, which is the same for
  // every tile.  Tiles that reach past the cache or the range take the
  // general path below.
  int voff[IPW];
#pragma unroll
  for (int u = 0; u < IPW; ++u) {
    const int ins = w * IPW + u, i = ins % IK;
    const int t = i * RPI + lane / CPR, pos = lane % CPR;
    voff[u] = (int)(((size_t)t * kstride + (size_t)((pos ^ RG::swz(t)) * EPC)) * sizeof(bf16));
  }
  const int cend = min(hi, P);  // keys below this come from the cache
  auto issue_fast = [&](int n, SpSlot<D>& sl) __attribute__((always_inline)) {
    const int j0 = lo + n * kTile;
    const bf16* kt = kc;
    const bf16* vt = vc;
    if constexpr (PAGED) {
      const int pi = j0 >> a.page_shift;
      const ptrdiff_t sh =
          ((ptrdiff_t)__builtin_amdgcn_readfirstlane(pages[pi - p0]) - pi) * ((ptrdiff_t)kstride << a.page_shift);
      kt += sh;
      vt += sh;
    }
    kt += (size_t)j0 * kstride;
    vt += (size_t)j0 * kstride;
    const int span = (int)((size_t)kTile * kstride * sizeof(bf16));
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(kt), 0, span, kBufferWord3);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(vt), 0, span, kBufferWord3);
#pragma unroll
    for (int u = 0; u < IPW; ++u) {
      const int ins = w * IPW + u, kv = ins / IK, i = ins % IK;
      bf16* dst = (kv == 0 ? sl.k : sl.v) + i * RPI * D;
      buf_to_lds16(kv == 0 ? rk : rv, dst, voff[u], 0);
    }
  };

  // This wave's copies of tile n (keys past the range read the range's last
  // key, in bounds, and are masked below).
  auto issue = [&](int n, SpSlot<D>& sl) __attribute__((always_inline)) {
    const int j0 = lo + n * kTile;
    if (j0 + kTile <= cend) {
      issue_fast(n, sl);
      return;
    }
    const bf16* kcb = kc;
    const bf16* vcb = vc;
    if constexpr (PAGED) {
      // the tile's rows (clamped to the range, all >= j0) lie in the page of
      // row j0: that page's base, shifted so that base + j * kstride is row j
      if (j0 < P) {
        const int pi = j0 >> a.page_shift;
        const ptrdiff_t sh = ((ptrdiff_t)pages[pi - p0] - pi) * ((ptrdiff_t)kstride << a.page_shift);
        kcb += sh;
        vcb += sh;
      }
    }
#pragma unroll
    for (int u = 0; u < IPW; ++u) {
      const int ins = w * IPW + u, kv = ins / IK, i = ins % IK;
      const int t = i * RPI + lane / CPR, pos = lane % CPR;
      const int j = min(j0 + t, hi - 1);
      const bf16* cb = kv == 0 ? kcb : vcb;
      const bf16* row = kv == 0 ? (j < P ? cb + (size_t)j * kstride : kbk + (size_t)(j - P) * kstride)
                                : (j < P ? cb + (size_t)j * kstride : vbk + (size_t)(j - P) * kstride);
      bf16* dst = (kv == 0 ? sl.k : sl.v) + i * RPI * D;
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void*)(row + (pos ^ RG::swz(t)) * EPC),
          (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
    }
  };

  // Scores and the running maximum m are kept in the log2 domain (scaled by
  // log2 e with 1/sqrt(d)), so each weight is one subtraction and one exp2;
  // m is converted back where it is written out for the combine.
  const float scale = 1.4426950408889634f / sqrtf((float)D);
  // The running sum of the weights comes from the MFMAs, as the product of
  // P^T with a tile of ones (every row of lsum holds it; only row 0 is kept
  // rescaled, the one that is read), so it is the sum of the same rounded
  // weights that enter P V.
  float m = -INFINITY;
  f32x16 acc[NCT], lsum = {};
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct) acc[ct] = f32x16{};
  op_t ones;
#pragma unroll
  for (int e = 0; e < E; ++e) ones[e] = (bf16)1.0f;

  auto compute = [&](int n, const SpSlot<D>& sl) __attribute__((always_inline)) {
    const int j0 = lo + n * kTile;
    f32x16 sc = {};
#pragma unroll
    for (int ks = 0; ks < KD; ++ks) {
      const int c = 2 * ks + hh;  // 16-byte chunk of elements ks*KW + hh*E
      sc = M::mma(load_op<bf16>(&sl.k[li * D + (c ^ RG::swz(li)) * EPC]), qop[ks], sc);
    }
    float p[16];
    if (j0 + kTile <= hi) {  // (uniform) a full tile needs no range masks
#pragma unroll
      for (int i = 0; i < 16; ++i) p[i] = sc[i] * scale;
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) p[i] = j0 + row_of(i, hh) < hi ? sc[i] * scale : -INFINITY;
    }
    float mt = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) mt = fmaxf(mt, p[i]);
    mt = fmaxf(mt, xor32(mt));
    const float mn = fmaxf(m, mt);
#pragma unroll
    for (int i = 0; i < 16; ++i) p[i] = __builtin_amdgcn_exp2f(p[i] - mn);
    if (__any(mn > m)) {
      const float corr = __builtin_amdgcn_exp2f(m - mn);
      lsum[0] *= corr;
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[ct][i] *= corr;
    }
    m = mn;
    // V^T operands by transposing reads: in each 16-lane quarter lane i
    // addresses key kb + i/4 at columns cb + 4*(i%4) .. +3 and receives
    // keys kb .. kb+3 of column cb + i.
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    const int qi = lane & 15;
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
      const int col = ct * kTile + 16 * ((lane >> 4) & 1) + 4 * (qi & 3);
#pragma unroll
      for (int ks = 0; ks < KL; ++ks) {
        auto piece = [&](int t) {
          const bf16* src = &sl.v[t * D + ((col / EPC) ^ RG::swz(t)) * EPC + col % EPC];
          return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)src);
        };
        const int kb = 16 * ks + 4 * hh + qi / 4;
        const s16x4 x0 = piece(kb), x1 = piece(kb + 8);
        const op_t va = __builtin_bit_cast(op_t, __builtin_shufflevector(x0, x1, 0, 1, 2, 3, 4, 5, 6, 7));
        acc[ct] = M::mma(va, cvt_op<bf16>(&p[ks * E]), acc[ct]);
      }
    }
#pragma unroll
    for (int ks = 0; ks < KL; ++ks) lsum = M::mma(ones, cvt_op<bf16>(&p[ks * E]), lsum);
  };

  // Wait for this wave's copies of tile n, with `later` tiles issued after
  // it still in flight.
  auto wait_tile = [&](int later) __attribute__((always_inline)) {
    if (later >= 2) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * IPW) : "memory");
    else if (later == 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(IPW) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  };
  auto slot = [&](auto S) -> SpSlot<D>& {
    if constexpr (decltype(S)::value == 0) return s0;
    else if constexpr (decltype(S)::value == 1) return s1;
    else if constexpr (decltype(S)::value == 2) return s2;
    else return s3;
  };
  auto step = [&](int n, auto S) __attribute__((always_inline)) {
    constexpr int SV = decltype(S)::value;
    wait_tile(min(R - 2, ntiles - 1 - n));
    lds_barrier_nodrain();  // tile n visible everywhere; slot of tile n-1 free
    if (n + R - 1 < ntiles) issue(n + R - 1, slot(std::integral_constant<int, (SV + R - 1) % R>{}));
    compute(n, slot(S));
  };

  if (0 < ntiles) issue(0, s0);
  if (1 < ntiles) issue(1, s1);
  if (2 < ntiles) issue(2, s2);
  for (int n = 0; n < ntiles; n += R) {
    step(n, std::integral_constant<int, 0>{});
    if (n + 1 < ntiles) step(n + 1, std::integral_constant<int, 1>{});
    if (n + 2 < ntiles) step(n + 2, std::integral_constant<int, 2>{});
    if (n + 3 < ntiles) step(n + 3, std::integral_constant<int, 3>{});
  }

  if (li >= L) return;
  const float l = lsum[0];
  if (ns == 1) {
    // one range: the result is final, normalised here (no combine launch)
    const float inv = 1.0f / l;
    const size_t ob = (((size_t)b * L + li) * Hq + h) * D;
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
      for (int i = 0; i < 16; i += 4) {
        const float o[4] = {acc[ct][i] * inv, acc[ct][i + 1] * inv, acc[ct][i + 2] * inv,
                            acc[ct][i + 3] * inv};
        store_out4<bf16>(a.out, ob + ct * kTile + row_of(i, hh), o, a.s.out_f32);
      }
    return;
  }
  const size_t row = (((size_t)b * Hq + h) * ns + s) * L + li;
  float* wacc = (float*)a.ws + row * D;
  float* wml = (float*)a.ws + (size_t)a.s.B * Hq * ns * L * D + row * 2;
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
    for (int i = 0; i < 16; i += 4)
      *reinterpret_cast<f32x4*>(wacc + ct * kTile + row_of(i, hh)) =
          f32x4{acc[ct][i], acc[ct][i + 1], acc[ct][i + 2], acc[ct][i + 3]};
  if (hh == 0) {
    wml[0] = m * 0.6931471805599453f;  // back to the natural log
    wml[1] = l;
  }
}

// Merge of the n_split partial results.  A thread handles 4 columns of one
// (request, head, query) row (16-byte loads); a workgroup of 256 threads
// covers 256 / (D/4) rows.
template <typename T, int D>
__global__ __launch_bounds__(256) void hyb_sp_combine_kernel(SoftmaxPrefixArgs a) {
  constexpr int TPR = D / 4;              // threads per row
  constexpr int RPB = 256 / TPR;          // rows per workgroup
  const int Hq = a.s.Hq, L = a.s.L, ns = a.n_split;
  const size_t nrows = (size_t)a.s.B * Hq * L;
  const size_t r = (size_t)blockIdx.x * RPB + threadIdx.x / TPR;
  if (r >= nrows) return;
  const int c = (threadIdx.x % TPR) * 4;
  const int i = (int)(r % L);
  const size_t bh = r / L;
  const int b = (int)(bh / Hq), h = (int)(bh % Hq);
  const size_t row0 = (bh * ns) * L + i;
  const float* wacc = (const float*)a.ws;
  const float* wml = wacc + (size_t)a.s.B * Hq * ns * L * D;
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, wml[(row0 + (size_t)s * L) * 2]);
  f32x4 num = {0.0f, 0.0f, 0.0f, 0.0f};
  float den = 0.0f;
  for (int s = 0; s < ns; ++s) {
    const size_t rr = row0 + (size_t)s * L;
    const float ms = wml[rr * 2];
    if (ms == -INFINITY) continue;
    const float wgt = expf(ms - M);
    const f32x4 x = *reinterpret_cast<const f32x4*>(wacc + rr * D + c);
#pragma unroll
    for (int e = 0; e < 4; ++e) num[e] += wgt * x[e];
    den += wgt * wml[rr * 2 + 1];
  }
  const float o[4] = {num[0] / den, num[1] / den, num[2] / den, num[3] / den};
  store_out4<T>(a.out, (((size_t)b * L + i) * Hq + h) * D + c, o, a.s.out_f32);
}

int softmax_prefix_splits(const Shape& s, int max_prefix) {
  const long units = (long)s.B * s.Hkv;
  long want = units > 0 ? (2048 + units - 1) / units : 1;
  const long cap = ((long)max_prefix + s.L + 511) / 512;
  if (want > cap) want = cap;
  // no range longer than kMaxRange keys (the paged kernel stages a range's
  // page numbers in LDS)
  const long least = ((long)max_prefix + s.L + kMaxRange - 1) / kMaxRange;
  if (want < least) want = least;
  if (want < 1) want = 1;
  return (int)want;
}

// A single KV range per (request, KV head) writes the normalised output
// directly and needs no workspace.
size_t softmax_prefix_ws_bytes(const Shape& s, int n_split) {
  if (n_split <= 1) return 0;
  return (size_t)s.B * s.Hq * n_split * s.L * (s.D + 2) * sizeof(float);
}

template <typename T, int D, bool PAGED>
static hipError_t sp_go(const SoftmaxPrefixArgs& a, hipStream_t st) {
  const int ns = a.n_split;
  int chunk = (a.max_prefix + a.s.L + ns - 1) / ns;
  chunk = (chunk + kTile - 1) / kTile * kTile;
  const int G = a.s.Hq / a.s.Hkv;
  const dim3 grid(a.s.B * a.s.Hkv * ns);
  bool launched_ring = false;
  if constexpr (sizeof(T) == 2) {
    launched_ring = true;
    switch (G) {
      case 1: hipLaunchKernelGGL((hyb_sp_ring_kernel<D, 1, PAGED>), grid, dim3(kWave), 0, st, a, chunk); break;
      case 2: hipLaunchKernelGGL((hyb_sp_ring_kernel<D, 2, PAGED>), grid, dim3(kWave * 2), 0, st, a, chunk); break;
      case 4: hipLaunchKernelGGL((hyb_sp_ring_kernel<D, 4, PAGED>), grid, dim3(kWave * 4), 0, st, a, chunk); break;
      case 8: hipLaunchKernelGGL((hyb_sp_ring_kernel<D, 8, PAGED>), grid, dim3(kWave * 8), 0, st, a, chunk); break;
      default: launched_ring = false;  // the register-staged kernel below
    }
  }
#define HYB_SP_CASE(NG)                                                               \
  case NG:                                                                            \
    hipLaunchKernelGGL((hyb_sp_partial_kernel<T, D, NG, PAGED>), grid, dim3(kWave * NG), 0, st, a, \
                       chunk);                                                        \
    break;
  if (!launched_ring) {
    switch (G) {
      HYB_SP_CASE(1)
      HYB_SP_CASE(2)
      HYB_SP_CASE(3)
      HYB_SP_CASE(4)
      HYB_SP_CASE(5)
      HYB_SP_CASE(6)
      HYB_SP_CASE(7)
      HYB_SP_CASE(8)
      default: return hipErrorInvalidValue;
    }
  }
#undef HYB_SP_CASE
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ns == 1) return e;  // one range: already written out
  {
    const size_t rows = (size_t)a.s.B * a.s.Hq * a.s.L;
    constexpr int RPB = 256 / (D / 4);
    hipLaunchKernelGGL((hyb_sp_combine_kernel<T, D>), dim3((unsigned)((rows + RPB - 1) / RPB)),
                       dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

template <bool PAGED>
static hipError_t sp_dispatch(const SoftmaxPrefixArgs& a, hipStream_t st) {
  if (a.s.dtype == 1)
    return a.s.D == 64 ? sp_go<bf16, 64, PAGED>(a, st) : sp_go<bf16, 128, PAGED>(a, st);
  return a.s.D == 64 ? sp_go<float, 64, PAGED>(a, st) : sp_go<float, 128, PAGED>(a, st);
}

hipError_t launch_softmax_prefix(const SoftmaxPrefixArgs& a, hipStream_t st) {
  if (a.s.Hq / a.s.Hkv > kMaxGroup) return hipErrorInvalidValue;
  if (a.page_table) {
    if (a.page_shift < 5 || a.n_pages < 1) return hipErrorInvalidValue;
    return sp_dispatch<true>(a, st);
  }
  return sp_dispatch<false>(a, st);
}

}  // namespace hyb
