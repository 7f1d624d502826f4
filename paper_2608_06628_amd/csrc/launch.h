// launch.h -- internal interface between the C-ABI layer (api.cpp) and the
// kernel translation units.  Arguments arrive here already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hyb {

struct Shape {
  int B, Hq, Hkv, D, L, F, dtype, n_slots;  // F = feat_dim / 2
  int out_f32;                              // out is fp32 whatever dtype is
  int step_kernel = 0;                      // step: 0 auto, 1 split, 2 whole, 3 halves
};

// block_len (nullable, device [B]): request b uses its first block_len[b]
// tokens of the L-token block (clamped to 0 .. L); the rest are padding.
struct StepArgs {
  Shape s;
  const void *q, *k, *v, *W;
  const float* alpha;
  const float *S, *z;
  const int32_t* slots;
  void* out;
  const int32_t* block_len;
};

struct CommitArgs {
  Shape s;
  const void *k, *v, *W;
  float *S, *z;
  const int32_t* slots;
  const int32_t* block_len;
};

struct PrefillArgs {
  Shape s;
  int T;
  const void *q, *k, *v, *W;
  const float* alpha;
  float *S, *z;
  const int32_t* slots;
  void* out;  // may be null
  float* ws;  // per-segment state deltas (nseg > 1), caller's workspace
};

// Backward of the block-causal hybrid layer over T tokens (empty starting
// state) with respect to W and alpha.  Exactly one of dout (upstream
// gradient) and target (teacher output: squared-error objective) is set.
struct BackwardArgs {
  Shape s;
  int T;
  const void *q, *k, *v, *W;
  const float* alpha;
  const void* dout;
  const void* target;
  float *dW, *dalpha, *loss;  // loss may be null
  void* ws;
  // Gradients with respect to the inputs (fp32, layouts of q, k, v), all
  // three set or all null; dk and dv are summed over the query heads that
  // share a KV head.
  float *dq = nullptr, *dk = nullptr, *dv = nullptr;
};

struct SoftmaxPrefixArgs {
  Shape s;
  const void *q, *k, *v, *k_cache, *v_cache;
  const int32_t* prefix_len;
  int max_prefix;
  void* out;
  void* ws;
  int n_split;  // KV splits per (request, KV head)
  // Paged cache (page_table non-null): k_cache, v_cache are page pools
  // [n_pages][1 << page_shift][Hkv][d]; cached token j of request b is row
  // j & (page size - 1) of page page_table[b * max_pages + (j >> page_shift)]
  // (clamped to the pool); max_prefix = max_pages << page_shift.
  const int32_t* page_table;
  int page_shift, max_pages, n_pages;
};

hipError_t launch_step(const StepArgs& a, hipStream_t st);
// The step for small batches: one wave per (request, head, 32-column slice).
hipError_t launch_step_small(const StepArgs& a, hipStream_t st);
// Whether the automatic choice takes the split kernel for these dims.
bool step_prefers_split(const Shape& s);
// The column-split step (two workgroups per group of four query heads, each
// streaming half of every head's state columns): whether a shape can take
// it, and whether the automatic choice does.
bool step_halves_supported(const Shape& s);
bool step_prefers_halves(const Shape& s);
// The step fused with the commit of the same block: S and z are updated in
// place after the step has read them (the StepArgs state pointers must be
// writable).
hipError_t launch_step_commit(const StepArgs& a, hipStream_t st);
// hybrid_state_commit with four query heads per workgroup sharing their K
// and V (bf16, f <= d, Hq / Hkv a multiple of 4, F <= 64; otherwise the
// per-head commit kernel).
bool commit_grouped_supported(const Shape& s);
hipError_t launch_commit_grouped(const CommitArgs& a, hipStream_t st);
hipError_t launch_commit(const CommitArgs& a, hipStream_t st);
hipError_t launch_prefill(const PrefillArgs& a, hipStream_t st);
hipError_t launch_softmax_prefix(const SoftmaxPrefixArgs& a, hipStream_t st);

// How a prompt of nblk blocks is cut for the segment scan: nseg walk
// segments of sb blocks (the last takes the rest), and the state increments
// of segments 0 .. nseg-2 computed in ppseg pieces of pb blocks per segment,
// npieces() in all (every piece non-empty).  Walk segment s starts from the
// incoming state plus pieces 0 .. s*ppseg - 1.
struct SegPlan {
  int nseg = 1, sb = 0, ppseg = 1, pb = 0;
  __host__ __device__ int npieces() const { return (nseg - 1) * ppseg; }
  __host__ __device__ int piece_lo(int pc) const { return (pc / ppseg) * sb + (pc % ppseg) * pb; }
  __host__ __device__ int piece_hi(int pc) const {
    const int hi = (pc / ppseg) * sb + (pc % ppseg + 1) * pb, end = (pc / ppseg + 1) * sb;
    return hi < end ? hi : end;
  }
};
// The prefill's plan (one round of walk workgroups over the chip, the
// increments in about as many workgroups), and the backward's (the same).
SegPlan prefill_plan(const Shape& s, int T);
SegPlan segment_plan(const Shape& s, int T);
// The prefill's workspace, and the part the increments take under a plan.
size_t prefill_ws_bytes(const Shape& s, int T);
size_t prefill_delta_ws_bytes(const Shape& s, const SegPlan& p);
// The increments alone: piece pc of the plan into a.ws (dS [units][npieces]
// [D][f], then dz [units][npieces][f]); a.S, a.z, a.q, a.alpha are not used.
hipError_t launch_prefill_delta(const PrefillArgs& a, const SegPlan& p, hipStream_t st);

// The library-held scratch buffer (scratch.hip) of the entry point that
// allocates nothing: its size, and its device address on the current device
// (looked up on the first call on each device).
constexpr size_t kScratchBytes = (size_t)64 << 20;
hipError_t scratch_device_ptr(void** ptr);

hipError_t launch_backward(const BackwardArgs& a, hipStream_t st);
bool backward_supported(const Shape& s);
// inputs: the workspace of a call that also forms dq, dk, dv
size_t backward_ws_bytes(const Shape& s, int T, bool inputs = false);

// Workspace of softmax_prefix_step for n_split splits.
size_t softmax_prefix_ws_bytes(const Shape& s, int n_split);
int softmax_prefix_splits(const Shape& s, int max_prefix);

}  // namespace hyb
