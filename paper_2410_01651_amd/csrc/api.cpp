// libgca C ABI: argument validation, workspace sizing and kernel dispatch.
// Nothing is launched unless every check passes; the library allocates nothing.
#include "gca.h"

#include <cmath>
#include <cstddef>
#include <cstdint>
#include <cstdlib>
#include <string>

#include "gca_plan.hpp"

namespace {

thread_local std::string g_last_error;

struct ProfileHook {
  hipEvent_t* events = nullptr;
  int capacity = 0;
  int count = 0;
  const char* names[4096];
};
thread_local ProfileHook g_profile;

gca_status fail(gca_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

gca_status from_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return GCA_OK;
  std::string msg = std::string(what) + ": " + hipGetErrorString(e);
  const char* kernel = gca::launch_error_kernel();
  if (kernel[0]) msg += std::string(" (kernel ") + kernel + ")";
  return fail(GCA_ERR_HIP, msg);
}

constexpr int64_t kMaxGrid = 2147483647;  // largest 1-D grid we launch

static_assert(GCA_NOALLOC_SCRATCH_BYTES == gca::kScratchBytes, "scratch size in the header and the library");

// the layout the Python binding mirrors
static_assert(sizeof(gca_problem) == 72 && offsetof(gca_problem, n_chunks) == 16 &&
                  offsetof(gca_problem, flags) == 56 && offsetof(gca_problem, gumbel_seed) == 64,
              "gca_problem layout");

gca_status check_problem(const gca_problem* p, gca::Shape& s) {
  if (!p) return fail(GCA_ERR_INVALID, "problem pointer is NULL");
  if (p->B < 1 || p->H < 1) return fail(GCA_ERR_INVALID, "B and H must be >= 1");
  if (p->d < 1 || p->S < 1) return fail(GCA_ERR_INVALID, "d and S must be >= 1");
  if (p->d != 64) return fail(GCA_ERR_UNSUPPORTED, "head dimension d must be 64");
  if (p->S != 64) return fail(GCA_ERR_UNSUPPORTED, "chunk size S must be 64");
  if (p->n_chunks < 1) return fail(GCA_ERR_INVALID, "n_chunks must be >= 1");
  if (p->n_chunks > 0x7fffffff) return fail(GCA_ERR_UNSUPPORTED, "n_chunks must fit in int32");
  if (p->topk < 1) return fail(GCA_ERR_INVALID, "topk must be >= 1");
  if (p->topk > 32) return fail(GCA_ERR_UNSUPPORTED, "topk must be <= 32");
  if (p->Hr != 1 && p->Hr != p->H) return fail(GCA_ERR_INVALID, "Hr must be 1 or H");
  if (p->D < 1) return fail(GCA_ERR_INVALID, "landmark width D must be >= 1");
  if (p->D % 64 != 0 || p->D > 8192) return fail(GCA_ERR_UNSUPPORTED, "D must be a multiple of 64, at most 8192");
  if (p->dtype != GCA_FP32 && p->dtype != GCA_BF16) return fail(GCA_ERR_INVALID, "unknown dtype");
  if (p->mode != GCA_CAUSAL && p->mode != GCA_DECODE) return fail(GCA_ERR_INVALID, "unknown mode");
  if (p->off_by_one != 0 && p->off_by_one != 1) return fail(GCA_ERR_INVALID, "off_by_one must be 0 or 1");
  if (!std::isfinite(p->score_scale) || !std::isfinite(p->attn_scale))
    return fail(GCA_ERR_INVALID, "scales must be finite");
  if (p->flags & ~(GCA_FLAG_FUSED_TOPK | GCA_FLAG_MATERIALIZE | GCA_FLAG_GUMBEL | GCA_FLAG_HOST_KV |
                   GCA_FLAG_LMK_ROW))
    return fail(GCA_ERR_INVALID, "unknown flag bits");
  if ((p->flags & GCA_FLAG_LMK_ROW) && p->mode != GCA_CAUSAL)
    return fail(GCA_ERR_UNSUPPORTED, "GCA_FLAG_LMK_ROW (S + 1 query rows) is supported in CAUSAL mode");
  if ((p->flags & GCA_FLAG_HOST_KV) && p->mode != GCA_DECODE)
    return fail(GCA_ERR_INVALID, "GCA_FLAG_HOST_KV is for DECODE mode");
  if ((p->flags & GCA_FLAG_FUSED_TOPK) && (p->flags & GCA_FLAG_MATERIALIZE))
    return fail(GCA_ERR_INVALID, "GCA_FLAG_FUSED_TOPK and GCA_FLAG_MATERIALIZE are exclusive");
  s.B = p->B;
  s.H = p->H;
  s.Hr = p->Hr;
  s.D = p->D;
  s.topk = p->topk;
  s.causal = p->mode == GCA_CAUSAL ? 1 : 0;
  s.nKV = p->n_chunks;
  s.nQ = s.causal ? p->n_chunks : 1;
  s.Sq = (p->flags & GCA_FLAG_LMK_ROW) ? gca::kChunk + 1 : gca::kChunk;
  s.bf16 = p->dtype == GCA_BF16 ? 1 : 0;
  s.off_by_one = p->off_by_one;
  s.score_scale = p->score_scale;
  s.attn_scale = p->attn_scale;
  s.gumbel = (p->flags & GCA_FLAG_GUMBEL) ? 1 : 0;
  s.gumbel_seed = p->gumbel_seed;
  const int64_t BH = (int64_t)s.B * s.H;
  if (BH > kMaxGrid / s.nQ || BH > kMaxGrid / s.nKV || (int64_t)s.B * s.Hr * s.nQ > kMaxGrid / s.topk)
    return fail(GCA_ERR_UNSUPPORTED, "problem too large for one launch");
  return GCA_OK;
}

// With GCA_FLAG_HOST_KV, k and v are pinned host allocations: the kernels use
// their device mapping.
gca_status device_view(const gca_problem* p, const void*& ptr, const char* name) {
  if (!(p->flags & GCA_FLAG_HOST_KV) || !ptr) return GCA_OK;
  // both: the runtime knows the allocation as pinned host memory, and it has a
  // device mapping
  hipPointerAttribute_t attr{};
  void* dev = nullptr;
  const hipError_t ea = hipPointerGetAttributes(&attr, ptr);
  const hipError_t e = ea == hipSuccess && attr.type == hipMemoryTypeHost
                           ? hipHostGetDevicePointer(&dev, const_cast<void*>(ptr), 0)
                           : hipErrorInvalidValue;
  if (e != hipSuccess || !dev) {
    (void)hipGetLastError();
    return fail(GCA_ERR_INVALID, std::string(name) + " is not pinned host memory with a device mapping "
                                                      "(GCA_FLAG_HOST_KV needs hipHostMalloc allocations)");
  }
  ptr = dev;
  return GCA_OK;
}

gca_status check_ptr(const void* ptr, const char* name, bool required, unsigned align) {
  if (!ptr) return required ? fail(GCA_ERR_INVALID, std::string(name) + " is NULL") : GCA_OK;
  if (reinterpret_cast<uintptr_t>(ptr) % align)
    return fail(GCA_ERR_INVALID, std::string(name) + " is not " + std::to_string(align) + "-byte aligned");
  return GCA_OK;
}

#define GCA_TRY(expr)               \
  do {                              \
    const gca_status st_ = (expr);  \
    if (st_ != GCA_OK) return st_;  \
  } while (0)

// Causal selection without the score matrix when asked to, or when the matrix
// would exceed 256 MiB (unless the caller insists on materialising it).
bool fused_path(const gca_problem* p, const gca::Shape& s) {
  if (p->flags & GCA_FLAG_FUSED_TOPK) return true;
  if (p->flags & GCA_FLAG_MATERIALIZE) return false;
  return sizeof(float) * (double)s.B * s.Hr * s.nQ * s.nKV > 256.0 * 1024 * 1024;
}

size_t forward_ws(const gca_problem* p, const gca::Shape& s) {
  if (!s.causal) return gca::decode_workspace(s);
  if (fused_path(p, s)) return gca::fused_workspace(s);
  return gca::align256(sizeof(float) * (size_t)s.B * s.Hr * s.nQ * s.nKV);
}

gca_status check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return GCA_OK;
  if (!ws) return fail(GCA_ERR_WORKSPACE, "workspace is NULL, need " + std::to_string(need) + " bytes");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(GCA_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (have < need)
    return fail(GCA_ERR_WORKSPACE,
                "workspace too small: " + std::to_string(have) + " < " + std::to_string(need) + " bytes");
  return GCA_OK;
}

}  // namespace

namespace gca {
thread_local hipError_t g_launch_error = hipSuccess;
thread_local const char* g_launch_error_kernel = "";
thread_local const char* g_reported_kernel = "";

bool profile_slot(const char* kernel, hipEvent_t* start, hipEvent_t* stop) {
  ProfileHook& h = g_profile;
  if (!h.events || 2 * (h.count + 1) > h.capacity) return false;
  h.names[h.count] = kernel;
  *start = h.events[2 * h.count];
  *stop = h.events[2 * h.count + 1];
  ++h.count;
  return true;
}

void note_launch_error(hipError_t e, const char* kernel) {
  if (e != hipSuccess && g_launch_error == hipSuccess) {
    g_launch_error = e;
    g_launch_error_kernel = kernel;
  }
}

hipError_t take_launch_error() {
  hipError_t e = g_launch_error;
  g_reported_kernel = g_launch_error_kernel;
  g_launch_error = hipSuccess;
  g_launch_error_kernel = "";
  if (e == hipSuccess) {
    e = hipGetLastError();
    g_reported_kernel = "";
  }
  return e;
}

const char* launch_error_kernel() { return g_reported_kernel; }

bool debug_sync() {
  static const bool on = [] {
    const char* v = std::getenv("GCA_DEBUG_SYNC");
    return v != nullptr && v[0] != '\0' && !(v[0] == '0' && v[1] == '\0');
  }();
  return on;
}
}  // namespace gca

extern "C" {

void gca_profile_arm(hipEvent_t* events, int capacity) {
  g_profile.events = capacity > 0 ? events : nullptr;
  g_profile.capacity = capacity > 0 ? (capacity < 4096 ? capacity : 4096) : 0;
  g_profile.count = 0;
}

int gca_profile_count(void) { return g_profile.count; }

const char* gca_profile_name(int i) {
  return (i >= 0 && i < g_profile.count && i < 4096) ? g_profile.names[i] : nullptr;
}


const char* gca_status_string(gca_status s) {
  switch (s) {
    case GCA_OK: return "GCA_OK";
    case GCA_ERR_INVALID: return "GCA_ERR_INVALID: malformed problem or argument";
    case GCA_ERR_UNSUPPORTED: return "GCA_ERR_UNSUPPORTED: outside the supported shapes";
    case GCA_ERR_WORKSPACE: return "GCA_ERR_WORKSPACE: workspace missing or too small";
    case GCA_ERR_HIP: return "GCA_ERR_HIP: a HIP launch failed";
  }
  return "unknown gca_status";
}

const char* gca_last_error(void) { return g_last_error.c_str(); }

size_t gca_workspace_size(const gca_problem* p, int op) {
  gca::Shape s;
  const std::string saved = g_last_error;
  if (check_problem(p, s) != GCA_OK) {
    g_last_error = saved;
    return 0;
  }
  if (op == GCA_OP_FORWARD) return forward_ws(p, s);
  if (op == GCA_OP_BACKWARD) return gca::bwd_workspace(s);
  return 0;
}

gca_status gca_chunk_scores(const gca_problem* p, const void* lmk_q, const void* lmk_k, float* scores,
                            hipStream_t stream) {
  gca::Shape s;
  GCA_TRY(check_problem(p, s));
  GCA_TRY(check_ptr(lmk_q, "lmk_q", true, 16));
  GCA_TRY(check_ptr(lmk_k, "lmk_k", true, 16));
  GCA_TRY(check_ptr(scores, "scores", true, 4));
  (void)hipGetLastError();
  (void)gca::take_launch_error();
  return from_hip(gca::launch_chunk_scores(s, lmk_q, lmk_k, scores, stream), "gca_chunk_scores");
}

gca_status gca_topk(const gca_problem* p, const float* scores, int32_t* idx, float* sel, hipStream_t stream) {
  gca::Shape s;
  GCA_TRY(check_problem(p, s));
  GCA_TRY(check_ptr(scores, "scores", true, 4));
  GCA_TRY(check_ptr(idx, "idx", true, 4));
  GCA_TRY(check_ptr(sel, "sel", true, 4));
  (void)hipGetLastError();
  (void)gca::take_launch_error();
  return from_hip(gca::launch_topk(s, scores, idx, sel, stream), "gca_topk");
}

gca_status gca_grouped_xattn_fwd(const gca_problem* p, const void* q, const void* k, const void* v,
                                 const int32_t* idx, const float* sel, void* out, float* lse, float* w,
                                 hipStream_t stream) {
  gca::Shape s;
  GCA_TRY(check_problem(p, s));
  GCA_TRY(check_ptr(q, "q", true, 16));
  GCA_TRY(check_ptr(k, "k", true, 16));
  GCA_TRY(check_ptr(v, "v", true, 16));
  GCA_TRY(check_ptr(idx, "idx", true, 4));
  GCA_TRY(check_ptr(sel, "sel", true, 4));
  GCA_TRY(check_ptr(out, "out", true, 16));
  GCA_TRY(check_ptr(lse, "lse", false, 4));
  GCA_TRY(check_ptr(w, "w", false, 4));
  GCA_TRY(device_view(p, k, "k"));
  GCA_TRY(device_view(p, v, "v"));
  (void)hipGetLastError();
  (void)gca::take_launch_error();
  return from_hip(gca::launch_xattn_fwd(s, q, k, v, idx, sel, out, lse, w, stream), "gca_grouped_xattn_fwd");
}

gca_status gca_grouped_xattn_bwd(const gca_problem* p, const void* q, const void* k, const void* v,
                                 const int32_t* idx, const float* sel, const float* lse, const void* dout,
                                 void* dq, void* dk, void* dv, float* dsel, const void* lmk_q, const void* lmk_k,
                                 float* dlmk_q, float* dlmk_k, void* workspace, size_t ws_bytes,
                                 hipStream_t stream) {
  gca::Shape s;
  GCA_TRY(check_problem(p, s));
  if (s.nQ * (int64_t)s.topk > 0x7fffffff) return fail(GCA_ERR_UNSUPPORTED, "nQ * topk must fit in int32");
  // the key-stationary pass packs (query chunk, slot) into one int
  if (s.nQ >= (int64_t(1) << 26)) return fail(GCA_ERR_UNSUPPORTED, "the backward takes fewer than 2^26 query chunks");
  GCA_TRY(check_ptr(q, "q", true, 16));
  GCA_TRY(check_ptr(k, "k", true, 16));
  GCA_TRY(check_ptr(v, "v", true, 16));
  GCA_TRY(check_ptr(idx, "idx", true, 4));
  GCA_TRY(check_ptr(sel, "sel", true, 4));
  GCA_TRY(check_ptr(lse, "lse", true, 4));
  GCA_TRY(check_ptr(dout, "dout", true, 16));
  GCA_TRY(check_ptr(dq, "dq", true, 16));
  GCA_TRY(check_ptr(dk, "dk", true, 16));
  GCA_TRY(check_ptr(dv, "dv", true, 16));
  GCA_TRY(check_ptr(dsel, "dsel", true, 4));
  GCA_TRY(check_ptr(dlmk_q, "dlmk_q", false, 4));
  GCA_TRY(check_ptr(dlmk_k, "dlmk_k", false, 4));
  GCA_TRY(check_ptr(lmk_q, "lmk_q", dlmk_k != nullptr, 16));
  GCA_TRY(check_ptr(lmk_k, "lmk_k", dlmk_q != nullptr, 16));
  GCA_TRY(check_ws(workspace, ws_bytes, gca::bwd_workspace(s)));
  GCA_TRY(device_view(p, k, "k"));
  GCA_TRY(device_view(p, v, "v"));
  (void)hipGetLastError();
  (void)gca::take_launch_error();
  return from_hip(gca::launch_xattn_bwd(s, q, k, v, idx, sel, lse, dout, dq, dk, dv, dsel, lmk_q, lmk_k, dlmk_q,
                                        dlmk_k, workspace, stream),
                  "gca_grouped_xattn_bwd");
}

// The forward path after validation: the selection (decode scan, single-pass
// select or score matrix + top-k) then the attention, on `workspace`.
static gca_status forward_dispatch(const gca_problem* p, const gca::Shape& s, const void* lmk_q, const void* lmk_k,
                                   const void* q, const void* k, const void* v, void* out, int32_t* idx,
                                   float* sel, float* lse, float* w, void* workspace, hipStream_t stream) {
  (void)hipGetLastError();
  (void)gca::take_launch_error();
  hipError_t e;
  if (!s.causal) {
    // decode: the scan leaves per-range lists; the attention merges them into
    // idx/sel and attends in the same launch
    e = gca::launch_decode_scan(s, lmk_q, lmk_k, workspace, stream);
    if (e != hipSuccess) return from_hip(e, "gca_forward (decode scan)");
    return from_hip(gca::launch_xattn_decode(s, gca::decode_list_scores(s, workspace),
                                             gca::decode_list_chunks(s, workspace), q, k, v, idx, sel, out, lse,
                                             w, lmk_q, lmk_k, stream),
                    "gca_forward (decode attention)");
  } else if (fused_path(p, s)) {
    e = gca::launch_fused_select(s, lmk_q, lmk_k, idx, sel, workspace, stream);
  } else {
    float* scores = reinterpret_cast<float*>(workspace);
    e = gca::launch_chunk_scores(s, lmk_q, lmk_k, scores, stream);
    if (e == hipSuccess) e = gca::launch_topk(s, scores, idx, sel, stream);
  }
  if (e != hipSuccess) return from_hip(e, "gca_forward (selection)");
  return from_hip(gca::launch_xattn_fwd(s, q, k, v, idx, sel, out, lse, w, stream), "gca_forward (attention)");
}

static gca_status check_forward_args(const gca_problem* p, gca::Shape& s, const void* lmk_q,
                                     const void* lmk_k, const void* q, const void* k, const void* v, void* out,
                                     int32_t* idx, float* sel, float* lse, float* w) {
  GCA_TRY(check_problem(p, s));
  GCA_TRY(check_ptr(lmk_q, "lmk_q", true, 16));
  GCA_TRY(check_ptr(lmk_k, "lmk_k", true, 16));
  GCA_TRY(check_ptr(q, "q", true, 16));
  GCA_TRY(check_ptr(k, "k", true, 16));
  GCA_TRY(check_ptr(v, "v", true, 16));
  GCA_TRY(check_ptr(out, "out", true, 16));
  GCA_TRY(check_ptr(idx, "idx", true, 4));
  GCA_TRY(check_ptr(sel, "sel", true, 4));
  GCA_TRY(check_ptr(lse, "lse", false, 4));
  GCA_TRY(check_ptr(w, "w", false, 4));
  return GCA_OK;
}

gca_status gca_forward(const gca_problem* p, const void* lmk_q, const void* lmk_k, const void* q, const void* k,
                       const void* v, void* out, int32_t* idx, float* sel, float* lse, float* w, void* workspace,
                       size_t ws_bytes, hipStream_t stream) {
  gca::Shape s;
  GCA_TRY(check_forward_args(p, s, lmk_q, lmk_k, q, k, v, out, idx, sel, lse, w));
  GCA_TRY(check_ws(workspace, ws_bytes, forward_ws(p, s)));
  GCA_TRY(device_view(p, k, "k"));
  GCA_TRY(device_view(p, v, "v"));
  return forward_dispatch(p, s, lmk_q, lmk_k, q, k, v, out, idx, sel, lse, w, workspace, stream);
}

gca_status gca_forward_noalloc(const gca_problem* p, const void* lmk_q, const void* lmk_k, const void* q,
                               const void* k, const void* v, void* out, int32_t* idx, float* sel, float* lse,
                               float* w, hipStream_t stream) {
  gca::Shape s;
  GCA_TRY(check_forward_args(p, s, lmk_q, lmk_k, q, k, v, out, idx, sel, lse, w));
  const size_t need = forward_ws(p, s);
  if (need > gca::kScratchBytes)
    return fail(GCA_ERR_UNSUPPORTED, "gca_forward_noalloc: the problem needs " + std::to_string(need) +
                                         " bytes of scratch, more than the " + std::to_string(gca::kScratchBytes) +
                                         " bytes the library holds per device; use gca_forward with a workspace");
  GCA_TRY(device_view(p, k, "k"));
  GCA_TRY(device_view(p, v, "v"));
  void* scratch = nullptr;
  if (need > 0) {
    hipError_t e = hipSuccess;
    scratch = gca::scratch_ptr(&e);
    if (!scratch) return from_hip(e != hipSuccess ? e : hipErrorInvalidSymbol, "gca_forward_noalloc (scratch address)");
  }
  return forward_dispatch(p, s, lmk_q, lmk_k, q, k, v, out, idx, sel, lse, w, scratch, stream);
}

}  // extern "C"
