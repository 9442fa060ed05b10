// Host-side launchers shared between the C ABI (api.cpp) and the kernel files.
// Every launcher enqueues on `stream` and returns the hipError_t of its last
// launch; shapes have been validated by the caller.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <tuple>
#include <utility>

namespace gca {

struct Shape {
  int B, H, Hr, D, topk;
  int64_t nQ;      // landmark query rows (query chunks)
  int64_t nKV;     // key/value chunks (score columns)
  int causal;      // 1: row t feeds chunk t+1 and sees chunks [0,t); 0: decode
  int bf16;        // element type of tensors: 1 bf16, 0 fp32
  int off_by_one;
  float score_scale, attn_scale;
  int gumbel;            // 1: Gumbel top-k selection
  uint64_t gumbel_seed;  // its generator seed
};

// Eq. 1 scores, written as a [B,Hr,nQ,nKV] fp32 matrix.
hipError_t launch_chunk_scores(const Shape& s, const void* lmk_q, const void* lmk_k, float* scores,
                               hipStream_t stream);
// Eq. 1 top-k over a score matrix.
hipError_t launch_topk(const Shape& s, const float* scores, int32_t* idx, float* sel,
                       hipStream_t stream);
// Decode selection, first half: a split scan of all past landmark keys (Eq. 1)
// that leaves, for every retrieval row, `lists` lists of the best k of `pw`
// chunks each (in the workspace; scan_list_of gives a chunk's list).  The decode
// attention merges them.
struct DecodePlan {
  int64_t pw;     // chunks per list (a quarter of one scan workgroup's contiguous range)
  int64_t lists;  // lists per retrieval row
  int64_t wgs;    // scan workgroups per row
};
DecodePlan decode_plan(const Shape& s);
size_t decode_workspace(const Shape& s);
float* decode_list_scores(const Shape& s, void* ws);
int* decode_list_chunks(const Shape& s, void* ws);
hipError_t launch_decode_scan(const Shape& s, const void* lmk_q, const void* lmk_k, void* ws, hipStream_t stream);
// Decode attention (Eq. 2-3 for the one query chunk of every (batch, head)).
// With lists (list_s != null) it first merges them into the row's top-k and
// writes idx/sel; without, idx/sel are its inputs.
// With Gumbel top-k the lists rank noisy scores and the chosen chunks' raw
// scores are recomputed from lmk_q / lmk_k (unused otherwise).
hipError_t launch_xattn_decode(const Shape& s, const float* list_s, const int* list_j, const void* q,
                               const void* k, const void* v, int32_t* idx, float* sel, void* out, float* lse,
                               float* w, const void* lmk_q, const void* lmk_k, hipStream_t stream);
// Causal: scores and top-k in one pass, no score matrix.
size_t fused_workspace(const Shape& s);
hipError_t launch_fused_select(const Shape& s, const void* lmk_q, const void* lmk_k, int32_t* idx,
                               float* sel, void* ws, hipStream_t stream);

// Eq. 2-3 forward.
hipError_t launch_xattn_fwd(const Shape& s, const void* q, const void* k, const void* v,
                            const int32_t* idx, const float* sel, void* out, float* lse, float* w,
                            hipStream_t stream);

// Backward (Algorithm 2 and the score/landmark chain rule).
size_t bwd_workspace(const Shape& s);
hipError_t launch_xattn_bwd(const Shape& s, const void* q, const void* k, const void* v,
                            const int32_t* idx, const float* sel, const float* lse, const void* dout,
                            void* dq, void* dk, void* dv, float* dsel, const void* lmk_q,
                            const void* lmk_k, float* dlmk_q, float* dlmk_k, void* ws,
                            hipStream_t stream);

// The per-kernel timing hook (gca_profile_arm): the next pair of the caller's
// events for `kernel`, or false when the hook is disarmed or full.
bool profile_slot(const char* kernel, hipEvent_t* start, hipEvent_t* stop);
// Keeps a launch's error (the first one of a sequence).
void note_launch_error(hipError_t e);
// The first launch error since the last call (hipSuccess if none); clears it.
hipError_t take_launch_error();

template <typename Tup, size_t... I>
inline void kernel_arg_ptrs(Tup& t, void** p, std::index_sequence<I...>) {
  ((p[I] = static_cast<void*>(&std::get<I>(t))), ...);
}

// Every kernel is launched through here.  The arguments are converted to the
// kernel's parameter types; while the timing hook is armed the dispatch itself
// carries a start and a stop event (hipExtLaunchKernel), so timing a kernel adds
// no packets to the stream and measures the kernel alone.
template <typename... KArgs, typename... Args>
inline void launch_kernel(const char* name, void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t smem,
                          hipStream_t stream, Args... args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "kernel argument count");
  std::tuple<KArgs...> a{static_cast<KArgs>(args)...};
  void* ptrs[sizeof...(KArgs)];
  kernel_arg_ptrs(a, ptrs, std::index_sequence_for<KArgs...>{});
  hipEvent_t start = nullptr, stop = nullptr;
  const void* f = reinterpret_cast<const void*>(kernel);
  if (profile_slot(name, &start, &stop))
    note_launch_error(hipExtLaunchKernel(f, grid, block, ptrs, smem, stream, start, stop, 0));
  else
    note_launch_error(hipLaunchKernel(f, grid, block, ptrs, smem, stream));
}

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
inline int64_t round8(int64_t n) { return (n + 7) & ~int64_t(7); }

}  // namespace gca
