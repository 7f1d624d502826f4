// api.cpp -- the C ABI of libhybattn: host-side validation, then dispatch to
// the kernel launchers.  Every check runs before any HIP call, so a rejected
// call enqueues nothing and touches no buffer.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <string>

#include "../../include/hybrid_attn.h"
#include "launch.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return HYB_OK;
}

size_t elem_bytes(int dtype) { return dtype == HYB_BF16 ? 2 : 4; }
size_t out_bytes(const hyb::Shape& s) { return s.out_f32 ? 4 : elem_bytes(s.dtype); }

// Shape checks common to every entry point.  need_state: the call reads a
// state pool.
int check_dims(const hyb_dims_t* d, bool need_state, hyb::Shape* s) {
  if (!d) return fail(HYB_ENULL, "dims is NULL");
  if (d->dtype != HYB_F32 && d->dtype != HYB_BF16)
    return fail(HYB_EDTYPE, "dtype %d is neither HYB_F32 nor HYB_BF16",
                d->dtype);
  if (d->batch < 0) return fail(HYB_EINVAL, "batch %d < 0", d->batch);
  if (d->n_q_heads < 1 || d->n_kv_heads < 1)
    return fail(HYB_EINVAL, "head counts must be >= 1 (Hq=%d, Hkv=%d)",
                d->n_q_heads, d->n_kv_heads);
  if (d->n_q_heads % d->n_kv_heads != 0)
    return fail(HYB_EINVAL, "n_kv_heads %d does not divide n_q_heads %d",
                d->n_kv_heads, d->n_q_heads);
  if (d->head_dim <= 0 || d->block <= 0 || d->feat_dim <= 0)
    return fail(HYB_EINVAL, "head_dim, block and feat_dim must be positive");
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(HYB_EUNSUPPORTED, "head_dim %d not supported (64 or 128)",
                d->head_dim);
  if (d->feat_dim != 64 && d->feat_dim != 128 && d->feat_dim != 256)
    return fail(HYB_EUNSUPPORTED,
                "feat_dim %d not supported (64, 128 or 256)", d->feat_dim);
  if (d->block > 32)
    return fail(HYB_EUNSUPPORTED, "block %d not supported (1..32)", d->block);
  if (need_state && d->batch > 0 && d->n_slots < 1)
    return fail(HYB_EINVAL, "n_slots %d < 1", d->n_slots);
  if ((long long)d->batch * d->n_q_heads > 0x7fffffffLL)
    return fail(HYB_EINVAL, "batch * n_q_heads exceeds the grid limit");
  if (d->flags & ~(HYB_OUT_F32 | HYB_STEP_SPLIT | HYB_STEP_WHOLE | HYB_STEP_HALVES))
    return fail(HYB_EINVAL, "unknown flags 0x%x", d->flags);
  {
    const int kf = d->flags & (HYB_STEP_SPLIT | HYB_STEP_WHOLE | HYB_STEP_HALVES);
    if (kf & (kf - 1))
      return fail(HYB_EINVAL, "more than one of HYB_STEP_SPLIT, HYB_STEP_WHOLE, HYB_STEP_HALVES");
  }
  *s = hyb::Shape{d->batch,    d->n_q_heads,    d->n_kv_heads,
                  d->head_dim, d->block,        d->feat_dim / 2,
                  d->dtype,    d->n_slots,      (d->flags & HYB_OUT_F32) ? 1 : 0};
  s->step_kernel = (d->flags & HYB_STEP_SPLIT)    ? 1
                   : (d->flags & HYB_STEP_WHOLE)  ? 2
                   : (d->flags & HYB_STEP_HALVES) ? 3
                                                  : 0;
  if (s->step_kernel == 3 && !hyb::step_halves_supported(*s))
    return fail(HYB_EUNSUPPORTED,
                "HYB_STEP_HALVES needs bf16, feat_dim <= 128 and n_q_heads / n_kv_heads a "
                "multiple of 4");
  return HYB_OK;
}

// The step-kernel flags belong to hybrid_attn_step alone.
int no_step_flags(const hyb_dims_t* d) {
  if (d && (d->flags & (HYB_STEP_SPLIT | HYB_STEP_WHOLE | HYB_STEP_HALVES)))
    return fail(HYB_EINVAL,
                "HYB_STEP_SPLIT / HYB_STEP_WHOLE / HYB_STEP_HALVES apply to hybrid_attn_step only");
  return HYB_OK;
}

int check_ptr(const void* p, const char* name, bool required = true) {
  if (!p) return required ? fail(HYB_ENULL, "%s is NULL", name) : HYB_OK;
  if (reinterpret_cast<uintptr_t>(p) & 15)
    return fail(HYB_EALIGN, "%s is not 16-byte aligned", name);
  return HYB_OK;
}

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

int launched(hipError_t e, const char* what) {
  if (e != hipSuccess)
    return fail(HYB_ELAUNCH, "%s launch failed: %s", what,
                hipGetErrorString(e));
  return ok();
}

#define TRY(x)               \
  do {                       \
    int _rc = (x);           \
    if (_rc != HYB_OK) return _rc; \
  } while (0)

}  // namespace

extern "C" {

int hybrid_attn_step(const hyb_dims_t* dims, const void* q, const void* k,
                     const void* v, const void* W, const float* alpha,
                     const float* S, const float* z, const int32_t* slots,
                     const int32_t* block_len, void* out, void* stream) {
  hyb::Shape s;
  TRY(check_dims(dims, true, &s));
  if (s.B == 0) return ok();
  TRY(check_ptr(q, "q"));
  TRY(check_ptr(k, "k"));
  TRY(check_ptr(v, "v"));
  TRY(check_ptr(W, "W"));
  TRY(check_ptr(alpha, "alpha"));
  TRY(check_ptr(S, "S"));
  TRY(check_ptr(z, "z"));
  TRY(check_ptr(slots, "slots", false));
  TRY(check_ptr(block_len, "block_len", false));
  TRY(check_ptr(out, "out"));
  const size_t es = elem_bytes(s.dtype), f = 2 * (size_t)s.F;
  const size_t nq = (size_t)s.B * s.L * s.Hq * s.D * es;
  const size_t no = (size_t)s.B * s.L * s.Hq * s.D * out_bytes(s);
  const size_t nkv = (size_t)s.B * s.L * s.Hkv * s.D * es;
  const size_t nS = (size_t)s.n_slots * s.Hq * f * s.D * 4;
  const size_t nz = (size_t)s.n_slots * s.Hq * f * 4;
  const size_t nW = (size_t)s.Hq * s.F * s.D * es;
  if (overlap(out, no, q, nq) || overlap(out, no, k, nkv) ||
      overlap(out, no, v, nkv) || overlap(out, no, W, nW) ||
      overlap(out, no, S, nS) || overlap(out, no, z, nz) ||
      overlap(out, no, alpha, (size_t)s.Hq * 4) ||
      overlap(out, no, slots, (size_t)s.B * 4) ||
      overlap(out, no, block_len, (size_t)s.B * 4))
    return fail(HYB_EINVAL, "out overlaps an input");
  hyb::StepArgs a{s, q, k, v, W, alpha, S, z, slots, out, block_len};
  (void)hipGetLastError();
  return launched(hyb::launch_step(a, (hipStream_t)stream), "step");
}

int hybrid_attn_step_commit(const hyb_dims_t* dims, const void* q,
                            const void* k, const void* v, const void* W,
                            const float* alpha, float* S, float* z,
                            const int32_t* slots, const int32_t* block_len,
                            void* out, void* stream) {
  hyb::Shape s;
  TRY(check_dims(dims, true, &s));
  TRY(no_step_flags(dims));
  if (s.B == 0) return ok();
  TRY(check_ptr(q, "q"));
  TRY(check_ptr(k, "k"));
  TRY(check_ptr(v, "v"));
  TRY(check_ptr(W, "W"));
  TRY(check_ptr(alpha, "alpha"));
  TRY(check_ptr(S, "S"));
  TRY(check_ptr(z, "z"));
  TRY(check_ptr(slots, "slots", false));
  TRY(check_ptr(block_len, "block_len", false));
  TRY(check_ptr(out, "out"));
  const size_t es = elem_bytes(s.dtype), f = 2 * (size_t)s.F;
  const size_t nq = (size_t)s.B * s.L * s.Hq * s.D * es;
  const size_t no = (size_t)s.B * s.L * s.Hq * s.D * out_bytes(s);
  const size_t nkv = (size_t)s.B * s.L * s.Hkv * s.D * es;
  const size_t nS = (size_t)s.n_slots * s.Hq * f * s.D * 4;
  const size_t nz = (size_t)s.n_slots * s.Hq * f * 4;
  const size_t nW = (size_t)s.Hq * s.F * s.D * es;
  // Everything the kernel writes (out, S, z) is disjoint from everything it
  // reads and from each other.
  struct Buf {
    const void* p;
    size_t n;
  };
  const Buf written[3] = {{out, no}, {S, nS}, {z, nz}};
  const Buf read_only[7] = {{q, nq},     {k, nkv},
                            {v, nkv},     {W, nW},
                            {alpha, (size_t)s.Hq * 4}, {slots, (size_t)s.B * 4},
                            {block_len, (size_t)s.B * 4}};
  for (int i = 0; i < 3; ++i) {
    for (const Buf& r : read_only)
      if (overlap(written[i].p, written[i].n, r.p, r.n))
        return fail(HYB_EINVAL, "an output (out, S or z) overlaps an input");
    for (int j = i + 1; j < 3; ++j)
      if (overlap(written[i].p, written[i].n, written[j].p, written[j].n))
        return fail(HYB_EINVAL, "out, S and z overlap");
  }
  hyb::StepArgs a{s, q, k, v, W, alpha, S, z, slots, out, block_len};
  (void)hipGetLastError();
  return launched(hyb::launch_step_commit(a, (hipStream_t)stream), "step_commit");
}

int hybrid_state_commit(const hyb_dims_t* dims, const void* k, const void* v,
                        const void* W, float* S, float* z,
                        const int32_t* slots, const int32_t* block_len,
                        void* stream) {
  hyb::Shape s;
  TRY(check_dims(dims, true, &s));
  TRY(no_step_flags(dims));
  if (s.B == 0) return ok();
  TRY(check_ptr(k, "k"));
  TRY(check_ptr(v, "v"));
  TRY(check_ptr(W, "W"));
  TRY(check_ptr(S, "S"));
  TRY(check_ptr(z, "z"));
  TRY(check_ptr(slots, "slots", false));
  TRY(check_ptr(block_len, "block_len", false));
  const size_t f = 2 * (size_t)s.F;
  const size_t nS = (size_t)s.n_slots * s.Hq * f * s.D * 4;
  const size_t nz = (size_t)s.n_slots * s.Hq * f * 4;
  if (overlap(S, nS, z, nz)) return fail(HYB_EINVAL, "S and z overlap");
  hyb::CommitArgs a{s, k, v, W, S, z, slots, block_len};
  (void)hipGetLastError();
  return launched(hyb::launch_commit(a, (hipStream_t)stream), "commit");
}

}  // extern "C"

namespace {

// Validation and dispatch of the prefill.  ws == nullptr with use_scratch:
// the workspace is the library-held scratch buffer.
int prefill_impl(const hyb_dims_t* dims, int32_t seq_len, const void* q,
                 const void* k, const void* v, const void* W,
                 const float* alpha, float* S, float* z, const int32_t* slots,
                 void* out, void* ws, size_t ws_bytes, bool use_scratch,
                 void* stream) {
  hyb::Shape s;
  TRY(check_dims(dims, true, &s));
  TRY(no_step_flags(dims));
  if (seq_len <= 0 || seq_len % s.L != 0)
    return fail(HYB_EINVAL, "seq_len %d is not a positive multiple of block %d",
                seq_len, s.L);
  if (s.B == 0) return ok();
  TRY(check_ptr(k, "k"));
  TRY(check_ptr(v, "v"));
  TRY(check_ptr(W, "W"));
  TRY(check_ptr(S, "S"));
  TRY(check_ptr(z, "z"));
  TRY(check_ptr(slots, "slots", false));
  TRY(check_ptr(out, "out", false));
  if (out) {
    TRY(check_ptr(q, "q"));
    TRY(check_ptr(alpha, "alpha"));
  }
  const size_t need = hybrid_workspace_bytes(dims, HYB_OP_PREFILL, seq_len);
  if (use_scratch) {
    if (need > hyb::kScratchBytes)
      return fail(HYB_EWORKSPACE,
                  "prefill needs %zu scratch bytes, more than the %zu "
                  "(HYB_NOALLOC_SCRATCH_BYTES) the library holds; use "
                  "hybrid_state_prefill with a workspace",
                  need, hyb::kScratchBytes);
  } else {
    if (need > 0 && (!ws || ws_bytes < need))
      return fail(HYB_EWORKSPACE, "prefill needs %zu workspace bytes, got %zu",
                  need, ws ? ws_bytes : (size_t)0);
    TRY(check_ptr(ws, "ws", false));
  }
  const size_t es = elem_bytes(s.dtype), f = 2 * (size_t)s.F;
  const size_t nq = (size_t)s.B * seq_len * s.Hq * s.D * es;
  const size_t no = (size_t)s.B * seq_len * s.Hq * s.D * out_bytes(s);
  const size_t nkv = (size_t)s.B * seq_len * s.Hkv * s.D * es;
  const size_t nS = (size_t)s.n_slots * s.Hq * f * s.D * 4;
  const size_t nz = (size_t)s.n_slots * s.Hq * f * 4;
  if (overlap(S, nS, z, nz)) return fail(HYB_EINVAL, "S and z overlap");
  if (out && (overlap(out, no, q, nq) || overlap(out, no, k, nkv) ||
              overlap(out, no, v, nkv) || overlap(out, no, S, nS) ||
              overlap(out, no, z, nz)))
    return fail(HYB_EINVAL, "out overlaps an input");
  if (need > 0 && (overlap(ws, need, S, nS) || overlap(ws, need, z, nz) ||
                   overlap(ws, need, k, nkv) || overlap(ws, need, v, nkv) ||
                   (out && (overlap(ws, need, out, no) || overlap(ws, need, q, nq)))))
    return fail(HYB_EINVAL, "the workspace overlaps an argument");
  (void)hipGetLastError();
  if (use_scratch && need > 0) {
    void* p = nullptr;
    const hipError_t e = hyb::scratch_device_ptr(&p);
    if (e != hipSuccess)
      return fail(HYB_ELAUNCH, "scratch buffer lookup failed: %s",
                  hipGetErrorString(e));
    ws = p;
  }
  hyb::PrefillArgs a{s, seq_len, q, k, v, W, alpha, S, z, slots, out, (float*)ws};
  return launched(hyb::launch_prefill(a, (hipStream_t)stream), "prefill");
}

}  // namespace

extern "C" {

int hybrid_state_prefill(const hyb_dims_t* dims, int32_t seq_len,
                         const void* q, const void* k, const void* v,
                         const void* W, const float* alpha, float* S, float* z,
                         const int32_t* slots, void* out, void* ws,
                         size_t ws_bytes, void* stream) {
  return prefill_impl(dims, seq_len, q, k, v, W, alpha, S, z, slots, out, ws,
                      ws_bytes, false, stream);
}

int hybrid_state_prefill_noalloc(const hyb_dims_t* dims, int32_t seq_len,
                                 const void* q, const void* k, const void* v,
                                 const void* W, const float* alpha, float* S,
                                 float* z, const int32_t* slots, void* out,
                                 void* stream) {
  return prefill_impl(dims, seq_len, q, k, v, W, alpha, S, z, slots, out,
                      nullptr, 0, true, stream);
}

}  // extern "C"

namespace {

// Validation and dispatch of the softmax-prefix step; !paged:
// contiguous cache [B][max_prefix][Hkv][d]; otherwise page pools
// [n_pages][page_size][Hkv][d] and a [B][max_pages] page table.
int softmax_prefix_impl(const hyb_dims_t* dims, const void* q, const void* k,
                        const void* v, const void* k_cache,
                        const void* v_cache, const int32_t* prefix_len,
                        int32_t max_prefix, bool paged,
                        const int32_t* page_table, int32_t n_pages,
                        int32_t page_size, int32_t max_pages, void* out,
                        void* ws, size_t ws_bytes, void* stream) {
  hyb::Shape s;
  TRY(check_dims(dims, false, &s));
  TRY(no_step_flags(dims));
  int page_shift = 0;
  if (paged) {
    if (max_pages < 0) return fail(HYB_EINVAL, "max_pages %d < 0", max_pages);
    if (page_size < 32 || page_size > (1 << 16) || (page_size & (page_size - 1)))
      return fail(HYB_EUNSUPPORTED,
                  "page_size %d not supported (a power of two, 32 .. 65536)",
                  page_size);
    while ((1 << page_shift) < page_size) ++page_shift;
    if ((long long)max_pages * page_size > 0x7fffffffLL - 64)
      return fail(HYB_EINVAL, "max_pages * page_size exceeds the index range");
    if (max_pages > 0 && n_pages < 1)
      return fail(HYB_EINVAL, "n_pages %d < 1", n_pages);
    max_prefix = max_pages * page_size;
  }
  if (max_prefix < 0)
    return fail(HYB_EINVAL, "max_prefix %d < 0", max_prefix);
  if (s.Hq / s.Hkv > 8)
    return fail(HYB_EUNSUPPORTED,
                "softmax_prefix_step supports up to 8 query heads per KV head");
  if (s.B == 0) return ok();
  TRY(check_ptr(q, "q"));
  TRY(check_ptr(k, "k"));
  TRY(check_ptr(v, "v"));
  TRY(check_ptr(out, "out"));
  TRY(check_ptr(prefix_len, "prefix_len"));
  if (max_prefix > 0) {
    TRY(check_ptr(k_cache, paged ? "k_pages" : "k_cache"));
    TRY(check_ptr(v_cache, paged ? "v_pages" : "v_cache"));
    if (paged) TRY(check_ptr(page_table, "page_table"));
  }
  const size_t need =
      hybrid_workspace_bytes(dims, HYB_OP_SOFTMAX_PREFIX, max_prefix);
  if (need > 0 && (!ws || ws_bytes < need))
    return fail(HYB_EWORKSPACE,
                "softmax_prefix_step needs %zu workspace bytes, got %zu", need,
                ws ? ws_bytes : (size_t)0);
  TRY(check_ptr(ws, "ws", false));
  const size_t es = elem_bytes(s.dtype);
  const size_t nq = (size_t)s.B * s.L * s.Hq * s.D * es;
  const size_t no = (size_t)s.B * s.L * s.Hq * s.D * out_bytes(s);
  const size_t nkv = (size_t)s.B * s.L * s.Hkv * s.D * es;
  const size_t nc = paged ? (size_t)n_pages * page_size * s.Hkv * s.D * es
                          : (size_t)s.B * max_prefix * s.Hkv * s.D * es;
  const size_t nt = paged ? (size_t)s.B * max_pages * 4 : 0;
  if (overlap(out, no, q, nq) || overlap(out, no, k, nkv) ||
      overlap(out, no, v, nkv) || overlap(out, no, k_cache, nc) ||
      overlap(out, no, v_cache, nc) || overlap(out, no, ws, need) ||
      overlap(out, no, prefix_len, (size_t)s.B * 4) ||
      overlap(out, no, page_table, nt))
    return fail(HYB_EINVAL, "out overlaps an input or the workspace");
  // the split kernels write the workspace while they read the inputs
  if (need > 0 && (overlap(ws, need, q, nq) || overlap(ws, need, k, nkv) ||
                   overlap(ws, need, v, nkv) || overlap(ws, need, k_cache, nc) ||
                   overlap(ws, need, v_cache, nc) ||
                   overlap(ws, need, prefix_len, (size_t)s.B * 4) ||
                   overlap(ws, need, page_table, nt)))
    return fail(HYB_EINVAL, "the workspace overlaps an input");
  hyb::SoftmaxPrefixArgs a{s,         q,   k,  v,
                           k_cache,   v_cache, prefix_len, max_prefix,
                           out,       ws,  hyb::softmax_prefix_splits(s, max_prefix),
                           paged && max_prefix > 0 ? page_table : nullptr,
                           page_shift, max_pages, n_pages};
  (void)hipGetLastError();
  return launched(hyb::launch_softmax_prefix(a, (hipStream_t)stream),
                  "softmax_prefix_step");
}

}  // namespace

extern "C" {

int softmax_prefix_step(const hyb_dims_t* dims, const void* q, const void* k,
                        const void* v, const void* k_cache,
                        const void* v_cache, const int32_t* prefix_len,
                        int32_t max_prefix, void* out, void* ws,
                        size_t ws_bytes, void* stream) {
  return softmax_prefix_impl(dims, q, k, v, k_cache, v_cache, prefix_len,
                             max_prefix, false, nullptr, 0, 0, 0, out, ws,
                             ws_bytes, stream);
}

int softmax_prefix_step_paged(const hyb_dims_t* dims, const void* q,
                              const void* k, const void* v,
                              const void* k_pages, const void* v_pages,
                              int32_t n_pages, int32_t page_size,
                              const int32_t* page_table, int32_t max_pages,
                              const int32_t* prefix_len, void* out, void* ws,
                              size_t ws_bytes, void* stream) {
  return softmax_prefix_impl(dims, q, k, v, k_pages, v_pages, prefix_len, 0,
                             true, page_table, n_pages, page_size, max_pages,
                             out, ws, ws_bytes, stream);
}

}  // extern "C"

namespace {

// Validation and dispatch of the backward; dq, dk, dv all null (the Stage-1
// gradient only) or all set (the input gradients as well).
int backward_impl(const hyb_dims_t* dims, int32_t seq_len, const void* q,
                  const void* k, const void* v, const void* W,
                  const float* alpha, const void* dout, const void* target,
                  float* dq, float* dk, float* dv, bool inputs, float* dW,
                  float* dalpha, float* loss, void* ws, size_t ws_bytes,
                  void* stream) {
  hyb::Shape s;
  TRY(check_dims(dims, false, &s));
  if (dims->flags != 0) return fail(HYB_EINVAL, "flags must be 0 for the backward");
  if (!hyb::backward_supported(s))
    return fail(HYB_EUNSUPPORTED, "backward supports feat_dim 64 or 128, not %d",
                2 * s.F);
  if (seq_len <= 0 || seq_len % s.L != 0)
    return fail(HYB_EINVAL, "seq_len %d is not a positive multiple of block %d",
                seq_len, s.L);
  if (s.B == 0) return ok();
  TRY(check_ptr(q, "q"));
  TRY(check_ptr(k, "k"));
  TRY(check_ptr(v, "v"));
  TRY(check_ptr(W, "W"));
  TRY(check_ptr(alpha, "alpha"));
  TRY(check_ptr(dout, "dout", false));
  TRY(check_ptr(target, "target", false));
  if ((dout == nullptr) == (target == nullptr))
    return fail(HYB_EINVAL, "exactly one of dout and target must be given");
  if (dout && loss) return fail(HYB_EINVAL, "loss needs a target");
  if (inputs) {
    TRY(check_ptr(dq, "dq"));
    TRY(check_ptr(dk, "dk"));
    TRY(check_ptr(dv, "dv"));
  }
  TRY(check_ptr(dW, "dW"));
  TRY(check_ptr(dalpha, "dalpha"));
  TRY(check_ptr(loss, "loss", false));
  const size_t need = hybrid_workspace_bytes(
      dims, inputs ? HYB_OP_BACKWARD_FULL : HYB_OP_BACKWARD, seq_len);
  if (!ws || ws_bytes < need)
    return fail(HYB_EWORKSPACE, "backward needs %zu workspace bytes, got %zu",
                need, ws ? ws_bytes : (size_t)0);
  TRY(check_ptr(ws, "ws"));
  const size_t es = elem_bytes(s.dtype);
  const size_t nq = (size_t)s.B * seq_len * s.Hq * s.D * es;
  const size_t nkv = (size_t)s.B * seq_len * s.Hkv * s.D * es;
  const size_t nW = (size_t)s.Hq * s.F * s.D * es;
  const size_t nq4 = (size_t)s.B * seq_len * s.Hq * s.D * 4;
  const size_t nkv4 = (size_t)s.B * seq_len * s.Hkv * s.D * 4;
  struct Buf {
    const void* p;
    size_t n;
  };
  const Buf written[7] = {{dW, (size_t)s.Hq * s.F * s.D * 4},
                          {dalpha, (size_t)s.Hq * 4},
                          {loss, (size_t)s.Hq * 4},
                          {ws, need},
                          {dq, nq4},
                          {dk, nkv4},
                          {dv, nkv4}};
  const Buf read_only[6] = {{q, nq},  {k, nkv}, {v, nkv}, {W, nW},
                            {alpha, (size_t)s.Hq * 4},
                            {dout ? dout : target, nq}};
  for (int i = 0; i < 7; ++i) {
    for (int j = i + 1; j < 7; ++j)
      if (overlap(written[i].p, written[i].n, written[j].p, written[j].n))
        return fail(HYB_EINVAL, "outputs or the workspace overlap each other");
    for (int j = 0; j < 6; ++j)
      if (overlap(written[i].p, written[i].n, read_only[j].p, read_only[j].n))
        return fail(HYB_EINVAL, "an output or the workspace overlaps an input");
  }
  hyb::BackwardArgs a{s, seq_len, q, k, v, W, alpha, dout, target,
                      dW, dalpha, loss, ws};
  if (inputs) {
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
  }
  (void)hipGetLastError();
  return launched(hyb::launch_backward(a, (hipStream_t)stream), "backward");
}

}  // namespace

extern "C" {

int hybrid_attn_backward(const hyb_dims_t* dims, int32_t seq_len,
                         const void* q, const void* k, const void* v,
                         const void* W, const float* alpha, const void* dout,
                         const void* target, float* dW, float* dalpha,
                         float* loss, void* ws, size_t ws_bytes, void* stream) {
  return backward_impl(dims, seq_len, q, k, v, W, alpha, dout, target, nullptr,
                       nullptr, nullptr, false, dW, dalpha, loss, ws, ws_bytes,
                       stream);
}

int hybrid_attn_backward_full(const hyb_dims_t* dims, int32_t seq_len,
                              const void* q, const void* k, const void* v,
                              const void* W, const float* alpha,
                              const void* dout, const void* target, float* dq,
                              float* dk, float* dv, float* dW, float* dalpha,
                              float* loss, void* ws, size_t ws_bytes,
                              void* stream) {
  return backward_impl(dims, seq_len, q, k, v, W, alpha, dout, target, dq, dk,
                       dv, true, dW, dalpha, loss, ws, ws_bytes, stream);
}

size_t hybrid_workspace_bytes(const hyb_dims_t* dims, int32_t op,
                              int32_t extent) {
  hyb::Shape s;
  const std::string saved = g_err;
  const int rc = check_dims(dims, false, &s);
  g_err = saved;
  if (rc != HYB_OK || extent < 0) return 0;
  switch (op) {
    case HYB_OP_STEP:
    case HYB_OP_COMMIT:
      return 0;
    case HYB_OP_PREFILL:
      if (extent == 0 || extent % s.L != 0) return 0;
      return hyb::prefill_ws_bytes(s, extent);
    case HYB_OP_SOFTMAX_PREFIX:
      return hyb::softmax_prefix_ws_bytes(
          s, hyb::softmax_prefix_splits(s, extent));
    case HYB_OP_BACKWARD:
    case HYB_OP_BACKWARD_FULL:
      if (extent == 0 || extent % s.L != 0 || !hyb::backward_supported(s)) return 0;
      return hyb::backward_ws_bytes(s, extent, op == HYB_OP_BACKWARD_FULL);
  }
  return 0;
}

const char* hybrid_last_error(void) { return g_err.c_str(); }

}  // extern "C"
