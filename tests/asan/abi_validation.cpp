// Drives every libgca entry point through its argument checks on the host (no
// GPU): malformed problems, NULL and misaligned pointers, missing or short
// workspaces, the scratch limit of the allocation-free forward, and well-formed
// calls that reach a (stubbed) launch.  Built with the sanitizers by the CPU test
// suite; prints OK and exits 0 when every status is the expected one.
#include <cstdio>
#include <cstring>
#include <vector>

#include "gca.h"

namespace gca {
int stub_launches();
}

static int g_fail = 0;
#define EXPECT(cond)                                                   \
  do {                                                                 \
    if (!(cond)) {                                                     \
      std::fprintf(stderr, "line %d: %s (%s)\n", __LINE__, #cond, gca_last_error()); \
      ++g_fail;                                                        \
    }                                                                  \
  } while (0)

static gca_problem base(int mode = GCA_CAUSAL) {
  gca_problem p;
  std::memset(&p, 0, sizeof p);
  p.B = 2; p.H = 4; p.d = 64; p.S = 64; p.n_chunks = 100; p.topk = 8; p.Hr = 1; p.D = 256;
  p.score_scale = 0.0625f; p.attn_scale = 0.125f; p.dtype = GCA_BF16; p.mode = mode;
  return p;
}

int main() {
  alignas(256) static unsigned char mem[1 << 16];
  void* A = mem;               // aligned stand-in for every device pointer (never dereferenced)
  void* M = mem + 4;           // misaligned
  float* F = reinterpret_cast<float*>(mem);
  int32_t* I = reinterpret_cast<int32_t*>(mem);

  // status strings and sizes
  for (int s = 0; s < 5; ++s) EXPECT(std::strncmp(gca_status_string((gca_status)s), "GCA_", 4) == 0);
  EXPECT(std::strstr(gca_status_string((gca_status)77), "unknown") != nullptr);
  gca_problem p = base();
  EXPECT(gca_workspace_size(&p, GCA_OP_FORWARD) > 0);
  EXPECT(gca_workspace_size(&p, GCA_OP_BACKWARD) > 0);
  EXPECT(gca_workspace_size(&p, 9) == 0);
  EXPECT(gca_workspace_size(nullptr, GCA_OP_FORWARD) == 0);
  gca_problem dec = base(GCA_DECODE);
  dec.n_chunks = 262144;
  EXPECT(gca_workspace_size(&dec, GCA_OP_FORWARD) > 0);

  // malformed problems are rejected by every entry point
  struct Bad { void (*edit)(gca_problem&); gca_status want; } bad[] = {
      {[](gca_problem& q) { q.B = 0; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.d = 32; }, GCA_ERR_UNSUPPORTED},
      {[](gca_problem& q) { q.S = 128; }, GCA_ERR_UNSUPPORTED},
      {[](gca_problem& q) { q.n_chunks = 0; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.n_chunks = (int64_t)1 << 40; }, GCA_ERR_UNSUPPORTED},
      {[](gca_problem& q) { q.topk = 0; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.topk = 33; }, GCA_ERR_UNSUPPORTED},
      {[](gca_problem& q) { q.Hr = 3; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.D = 100; }, GCA_ERR_UNSUPPORTED},
      {[](gca_problem& q) { q.dtype = 5; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.mode = 2; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.off_by_one = 2; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.score_scale = 1.f / 0.f; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.flags = 64; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.flags = GCA_FLAG_FUSED_TOPK | GCA_FLAG_MATERIALIZE; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.flags = GCA_FLAG_HOST_KV; }, GCA_ERR_INVALID},
      {[](gca_problem& q) { q.B = 1 << 20; q.H = 1 << 10; }, GCA_ERR_UNSUPPORTED},
  };
  std::vector<unsigned char> ws(1 << 24);
  void* W = reinterpret_cast<void*>((reinterpret_cast<uintptr_t>(ws.data()) + 255) & ~uintptr_t(255));
  const size_t WB = ws.size() - 256;
  for (const Bad& b : bad) {
    gca_problem q = base();
    b.edit(q);
    EXPECT(gca_chunk_scores(&q, A, A, F, nullptr) == b.want);
    EXPECT(gca_topk(&q, F, I, F, nullptr) == b.want);
    EXPECT(gca_grouped_xattn_fwd(&q, A, A, A, I, F, A, F, F, nullptr) == b.want);
    EXPECT(gca_grouped_xattn_bwd(&q, A, A, A, I, F, F, A, A, A, A, F, A, A, F, F, W, WB, nullptr) == b.want);
    EXPECT(gca_forward(&q, A, A, A, A, A, A, I, F, F, F, W, WB, nullptr) == b.want);
    EXPECT(gca_forward_noalloc(&q, A, A, A, A, A, A, I, F, F, F, nullptr) == b.want);
    EXPECT(gca_workspace_size(&q, GCA_OP_FORWARD) == 0);
    EXPECT(std::strlen(gca_last_error()) > 0);
  }
  EXPECT(gca_forward(nullptr, A, A, A, A, A, A, I, F, F, F, W, WB, nullptr) == GCA_ERR_INVALID);

  // NULL and misaligned pointers
  EXPECT(gca_forward(&p, nullptr, A, A, A, A, A, I, F, F, F, W, WB, nullptr) == GCA_ERR_INVALID);
  EXPECT(gca_forward(&p, A, A, M, A, A, A, I, F, F, F, W, WB, nullptr) == GCA_ERR_INVALID);
  EXPECT(std::strstr(gca_last_error(), "aligned") != nullptr);
  EXPECT(gca_grouped_xattn_fwd(&p, A, A, A, I, F, nullptr, F, F, nullptr) == GCA_ERR_INVALID);
  EXPECT(gca_grouped_xattn_bwd(&p, A, A, A, I, F, nullptr, A, A, A, A, F, A, A, F, F, W, WB, nullptr) ==
         GCA_ERR_INVALID);
  // landmark gradients need the other side's landmarks
  EXPECT(gca_grouped_xattn_bwd(&p, A, A, A, I, F, F, A, A, A, A, F, A, nullptr, F, nullptr, W, WB, nullptr) ==
         GCA_ERR_INVALID);

  // workspaces
  const size_t need_f = gca_workspace_size(&p, GCA_OP_FORWARD), need_b = gca_workspace_size(&p, GCA_OP_BACKWARD);
  EXPECT(need_f <= WB && need_b <= WB);
  EXPECT(gca_forward(&p, A, A, A, A, A, A, I, F, F, F, nullptr, 0, nullptr) == GCA_ERR_WORKSPACE);
  EXPECT(gca_forward(&p, A, A, A, A, A, A, I, F, F, F, W, need_f - 1, nullptr) == GCA_ERR_WORKSPACE);
  EXPECT(gca_forward(&p, A, A, A, A, A, A, I, F, F, F, static_cast<char*>(W) + 16, need_f, nullptr) ==
         GCA_ERR_WORKSPACE);
  EXPECT(gca_grouped_xattn_bwd(&p, A, A, A, I, F, F, A, A, A, A, F, A, A, F, F, W, need_b - 1, nullptr) ==
         GCA_ERR_WORKSPACE);

  // the allocation-free forward's limit: a 4,096^2 score matrix is 64 MiB
  gca_problem big = base();
  big.B = 1; big.n_chunks = 4096; big.flags = GCA_FLAG_MATERIALIZE;
  EXPECT(gca_workspace_size(&big, GCA_OP_FORWARD) > GCA_NOALLOC_SCRATCH_BYTES);
  EXPECT(gca_forward_noalloc(&big, A, A, A, A, A, A, I, F, F, F, nullptr) == GCA_ERR_UNSUPPORTED);

  // nothing above reached a launch; well-formed calls do (and report the stub's failure)
  EXPECT(gca::stub_launches() == 0);
  EXPECT(gca_chunk_scores(&p, A, A, F, nullptr) == GCA_ERR_HIP);
  EXPECT(gca_topk(&p, F, I, F, nullptr) == GCA_ERR_HIP);
  EXPECT(gca_grouped_xattn_fwd(&p, A, A, A, I, F, A, F, F, nullptr) == GCA_ERR_HIP);
  EXPECT(gca_grouped_xattn_bwd(&p, A, A, A, I, F, F, A, A, A, A, F, A, A, F, F, W, need_b, nullptr) == GCA_ERR_HIP);
  EXPECT(gca_forward(&p, A, A, A, A, A, A, I, F, F, F, W, need_f, nullptr) == GCA_ERR_HIP);
  EXPECT(gca_forward_noalloc(&p, A, A, A, A, A, A, I, F, F, F, nullptr) == GCA_ERR_HIP);
  EXPECT(gca_forward(&dec, A, A, A, A, A, A, I, F, F, F, W, WB, nullptr) == GCA_ERR_HIP);
  EXPECT(gca::stub_launches() == 7);

  // the profiling hook clamps its capacity and reports nothing while disarmed
  gca_profile_arm(nullptr, 0);
  EXPECT(gca_profile_count() == 0);
  EXPECT(gca_profile_name(0) == nullptr);

  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("OK\n");
  return 0;
}
