// Host-side contract between the C ABI (api.cpp) and the kernel files: the
// validated problem shape, workspace plans, and the launchers each kernel file
// provides.  Host C++ only (no device code), so the ABI layer also builds with a
// plain host compiler.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace gca {

constexpr int kChunk = 64;  // tokens per chunk (S) and head dimension (d) supported

struct Shape {
  int B, H, Hr, D, topk;
  int64_t nQ;      // landmark query rows (query chunks)
  int64_t nKV;     // key/value chunks (score columns)
  int Sq;          // query rows per chunk: kChunk, or kChunk + 1 with the LMK row (causal only)
  int causal;      // 1: row t feeds chunk t+1 and sees chunks [0,t); 0: decode
  int bf16;        // element type of tensors: 1 bf16, 0 fp32
  int off_by_one;
  float score_scale, attn_scale;
  int gumbel;            // 1: Gumbel top-k selection
  uint64_t gumbel_seed;  // its generator seed
};

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
inline int64_t round8(int64_t n) { return (n + 7) & ~int64_t(7); }

// Compute units of the calling thread's current device (queried once per
// device).  Persistent kernels size their grids from it.
int device_cus();

// ------------------------------------------------------------ plans ----

// Decode selection: a split scan of all past landmark keys (Eq. 1) leaves, for
// every retrieval row, `lists` lists of the best k of `pw` chunks each; the
// decode attention merges them.  The plan does not depend on the device (the
// workspace size must not), so it targets 256 scan workgroups in all.
struct DecodePlan {
  int64_t pw;     // chunks per list (a quarter of one scan workgroup's contiguous range)
  int64_t lists;  // lists per retrieval row
  int64_t wgs;    // scan workgroups per row
};
DecodePlan decode_plan(const Shape& s);
size_t decode_workspace(const Shape& s);
float* decode_list_scores(const Shape& s, void* ws);
int* decode_list_chunks(const Shape& s, void* ws);

// Causal selection without the score matrix: blocks of kSelRows landmark rows
// against tiles of kSelTile key chunks.  Key tile j belongs to class j mod 8 (one
// class per XCD); a block's tiles of one class are split into parts of at most
// `tiles_per_part` tiles, and every (block, class, part) work item leaves the
// best k of its candidates for each of its rows.  A row has at most `lists`
// such lists (list number = class * parts_max + part).
constexpr int kSelRows = 128;
constexpr int kSelTile = 32;
constexpr int kSelClasses = 8;
struct SelectPlan {
  bool split;            // the split form applies (else one pass per row block, no workspace)
  int64_t blocks;        // row blocks per (batch, retrieval head)
  int64_t tiles;         // key tiles
  int tiles_per_part;
  int64_t parts_max;     // parts of one class in the largest row block
  int64_t lists;         // lists per row = kSelClasses * parts_max
  int64_t items_per_class;  // work items of one class per (batch, retrieval head)
};
SelectPlan select_plan(const Shape& s);
size_t fused_workspace(const Shape& s);

// Backward workspace: fusion weights, per-(token, slot) values of the
// query-stationary pass, dw partials and the inverse index (CSR) of the
// retrieval lists.  kHeadInts ints per key chunk: [0] offset of its list, [1]
// its length, [2 .. 2 + kHeadEntries) its first entries.
constexpr int kHeadInts = 16;
constexpr int kHeadEntries = 8;
struct BwdWs {
  float* w;        // [B*Hr, nQ, K] fusion weights
  float* Dbuf;     // [B*H, K, Lq]  -D_s per query token (slot-major: one slot's tokens contiguous; Lq = nQ * Sq)
  float* Lbuf;     // [B*H, K, Lq]  log2(e) lse - log2(w_s)
  float* dwp;      // [B*H, nQ, K, 2] dw partials per head and query half
  int* counts;     // [B*Hr, nKV]
  int* cursor;     // [B*Hr, nKV]
  int* offs;       // [B*Hr, nKV+1]
  int* unsorted;   // [B*Hr, nQ*K]
  int* sorted;     // [B*Hr, nQ*K]
  int* head;       // [B*Hr, nKV, kHeadInts]
};
BwdWs bwd_carve(const Shape& s, void* base);
size_t bwd_workspace(const Shape& s);

// ------------------------------------------------------- launchers ----
// Every launcher enqueues on `stream` and returns the hipError_t of its launches;
// shapes have been validated by the caller.

// Eq. 1 scores, written as a [B,Hr,nQ,nKV] fp32 matrix.
hipError_t launch_chunk_scores(const Shape& s, const void* lmk_q, const void* lmk_k, float* scores,
                               hipStream_t stream);
// Eq. 1 top-k over a score matrix.
hipError_t launch_topk(const Shape& s, const float* scores, int32_t* idx, float* sel, hipStream_t stream);
hipError_t launch_decode_scan(const Shape& s, const void* lmk_q, const void* lmk_k, void* ws, hipStream_t stream);
// Decode attention (Eq. 2-3 for the one query chunk of every (batch, head)).
// With lists (list_s != null) it first merges them into the row's top-k and
// writes idx/sel; without, idx/sel are its inputs.
// With Gumbel top-k the lists rank noisy scores and the chosen chunks' raw
// scores are recomputed from lmk_q / lmk_k (unused otherwise).
hipError_t launch_xattn_decode(const Shape& s, const float* list_s, const int* list_j, const void* q,
                               const void* k, const void* v, int32_t* idx, float* sel, void* out, float* lse,
                               float* w, const void* lmk_q, const void* lmk_k, hipStream_t stream);
// Causal: scores and top-k without the score matrix (workspace: fused_workspace),
// split over key-tile parts when select_plan(s).split ...
hipError_t launch_fused_select(const Shape& s, const void* lmk_q, const void* lmk_k, int32_t* idx,
                               float* sel, void* ws, hipStream_t stream);
// ... else one pass per 64-row block (no workspace).
hipError_t launch_fused_rowblocks(const Shape& s, const void* lmk_q, const void* lmk_k, int32_t* idx,
                                  float* sel, hipStream_t stream);
// Eq. 2-3 forward.
hipError_t launch_xattn_fwd(const Shape& s, const void* q, const void* k, const void* v,
                            const int32_t* idx, const float* sel, void* out, float* lse, float* w,
                            hipStream_t stream);
// Backward (Algorithm 2 and the score/landmark chain rule).
hipError_t launch_xattn_bwd(const Shape& s, const void* q, const void* k, const void* v,
                            const int32_t* idx, const float* sel, const float* lse, const void* dout,
                            void* dq, void* dk, void* dv, float* dsel, const void* lmk_q,
                            const void* lmk_k, float* dlmk_q, float* dlmk_k, void* ws,
                            hipStream_t stream);

// The per-kernel timing hook (gca_profile_arm): the next pair of the caller's
// events for `kernel`, or false when the hook is disarmed or full.
bool profile_slot(const char* kernel, hipEvent_t* start, hipEvent_t* stop);
// Keeps a launch's error (the first one of a sequence) and the kernel it came from.
void note_launch_error(hipError_t e, const char* kernel);
// The first launch error since the last call (hipSuccess if none); clears it.
hipError_t take_launch_error();
// The kernel named with the error take_launch_error() last returned ("" if none).
const char* launch_error_kernel();
// GCA_DEBUG_SYNC set in the environment (read once): every launch is followed
// by a stream synchronisation and an error check naming the kernel.
bool debug_sync();

// The allocation-free forward's device scratch array: this device's address of
// it (looked up once per device), or null with the HIP error in *err.
constexpr size_t kScratchBytes = size_t(16) << 20;
void* scratch_ptr(hipError_t* err);

}  // namespace gca
