// Grouped cross attention forward (Eq. 2-3 of the method; Algorithm 1 in the
// appendix is its tiled form).
//
// One workgroup of two waves per (batch, head, query chunk).  Each wave owns 32
// of the chunk's 64 query tokens and keeps their Q fragments in registers for
// the whole kernel.  The retrieved chunks' keys and values stream through a
// ring of LDS slots filled by asynchronous direct-to-LDS copies, several
// chunks ahead of the one being computed.  For every slot the workgroup
// computes S^T = K Q^T on the
// matrix cores, takes each query's softmax over the 64 keys (one retrieved
// chunk is exactly one tile, so no running rescale is needed), folds the
// fusion weight w_s / l_s into P, and accumulates O^T += V^T (w_s P_s)^T into a
// single fp32 accumulator shared by all slots.  The per-chunk outputs O'_s of
// Algorithm 1 are never written; the log-sum-exp of every (row, slot) is.
//
// Computing the transposed products keeps every query's statistics inside one
// lane (query = accumulator column): the softmax needs one cross-lane step, and
// the probability tile feeds the PV product straight from registers.  V^T
// fragments come from the row-major V tile through LDS transpose reads.
#include "gca_device.hpp"
#include "gca_launch.hpp"

#include <type_traits>

namespace gca {
namespace {

constexpr int kThreads = 128;

template <typename T> struct LdsLd;
template <> struct LdsLd<__bf16> { static constexpr int v = 72; };  // 144-byte rows
template <> struct LdsLd<float> { static constexpr int v = 68; };   // 272-byte rows

struct FwdParams {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* idx;
  const float* sel;
  void* out;
  float* lse;
  float* w;
  int H, Hr, topk;
  int64_t nQ, nKV, nwork;
  int causal;
  float attn_scale;
};

// LDS ring depth (retrieved chunks in flight per workgroup).
template <typename T> struct RingDepth;
template <> struct RingDepth<__bf16> { static constexpr int v = 4; };  // 4 x 16 KB
template <> struct RingDepth<float> { static constexpr int v = 2; };   // 2 x 32 KB

template <typename T, bool OBO>
__global__ __launch_bounds__(kThreads) void xattn_fwd_kernel(FwdParams p) {
  constexpr int NB = RingDepth<T>::v;
  constexpr int TILE = kS * kD;
  constexpr int L = Swz<T>::kCPR;  // copies per wave per slot: 2 tiles x kCPR / 2 waves
  // one LDS variable per ring slot: with the slot known at compile time in the
  // unrolled loop below, the compiler waits only for that slot's copies
  __shared__ __attribute__((aligned(16))) T ring0[2 * TILE];
  __shared__ __attribute__((aligned(16))) T ring1[2 * TILE];
  __shared__ __attribute__((aligned(16))) T ring2[NB > 2 ? 2 * TILE : 8];
  __shared__ __attribute__((aligned(16))) T ring3[NB > 3 ? 2 * TILE : 8];
  __shared__ float sLse[32 * kS];  // [slot][query]
  __shared__ float sW[32];
  __shared__ int sJ[32];
  __shared__ int sSlot[32];
  __shared__ int sN;

  const int64_t wid = xcd_swizzle(blockIdx.x, gridDim.x);
  if (wid >= p.nwork) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5;
  const int64_t c = wid % p.nQ;
  const int64_t bh = wid / p.nQ;
  const int h = (int)(bh % p.H);
  const int64_t b = bh / p.H;
  const int hr = p.Hr == 1 ? 0 : h;
  const int64_t t = p.causal ? c - 1 : 0;
  const int K = p.topk;
  const int64_t row_base = (b * p.Hr + hr) * p.nQ;  // retrieval rows of (b, hr)

  // The retrieval row's slots (Eq. 2 weights, compacted list of valid slots) by
  // wave 0 with one load per slot; wave 1 writes the weights of the causal last
  // row, which feeds no chunk and is owned by chunk 0.
  if (wave == 0 || (p.w && p.causal && c == 0 && (p.Hr != 1 || h == 0))) {
    const int64_t row = wave == 0 ? t : p.nQ - 1;
    float wv = 0.f;
    int jv = -1;
    const bool any = row >= 0 && wave_row_weight(p.idx, p.sel, (row_base + row) * K, K, p.nKV, wv, jv);
    if (wave == 0) {
      const uint64_t mask = __ballot(jv >= 0 && lane < K);
      if (lane < 32) {
        sW[lane] = wv;
        sJ[lane] = jv;
      }
      if (jv >= 0 && lane < K) sSlot[__popcll(mask & ((1ull << lane) - 1))] = lane;
      if (lane == 0) sN = any ? __popcll(mask) : 0;
      // this row's weights go out with the chunk it feeds
      if (p.w && row >= 0 && lane < K && (p.Hr != 1 || h == 0)) p.w[(row_base + row) * K + lane] = wv;
    } else if (lane < K) {
      p.w[(row_base + row) * K + lane] = wv;
    }
  }
  __syncthreads();
  const int n = sN;

  const int64_t tok0 = ((b * p.H + h) * p.nQ + c) * kS;  // first query token of the chunk
  T* out = reinterpret_cast<T*>(p.out) + tok0 * kD;
  float* lse = p.lse ? p.lse + tok0 * K : nullptr;

  if (n == 0) {
    for (int e = tid; e < kS * kD / 4; e += kThreads) store4(out + 4 * e, 0.f, 0.f, 0.f, 0.f);
    if (lse)
      for (int e = tid; e < kS * K; e += kThreads) lse[e] = -INFINITY;
    return;
  }

  const int qi = 32 * wave + (lane & 31);  // this lane's query token within the chunk
  const T* qrow = reinterpret_cast<const T*>(p.q) + (tok0 + qi) * kD;
  Frag<T> qf[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) qf[kb] = load_frag(qrow + 16 * kb + 8 * hh);
  wait_vmem<0>();  // nothing but the chunk copies may be pending inside the slot loop

  const int64_t kv0 = (b * p.H + h) * p.nKV * TILE;
  const T* kbase = reinterpret_cast<const T*>(p.k) + kv0;
  const T* vbase = reinterpret_cast<const T*>(p.v) + kv0;
  auto slot_buf = [&](auto B) __device__ -> T* {
    constexpr int b = decltype(B)::value;
    if constexpr (b == 0) return ring0;
    else if constexpr (b == 1) return ring1;
    else if constexpr (b == 2) return ring2;
    else return ring3;
  };
  auto issue = [&](auto B, int u) __device__ {
    const int64_t j = sJ[sSlot[u]];
    T* dst = slot_buf(B);
    dma_tile<T, 2>(kbase + j * TILE, dst, wave, lane);
    dma_tile<T, 2>(vbase + j * TILE, dst + TILE, wave, lane);
  };
  issue(std::integral_constant<int, 0>{}, 0);
  if (NB > 2 && n > 1) issue(std::integral_constant<int, 1>{}, 1);
  if (NB > 3 && n > 2) issue(std::integral_constant<int, (NB > 3 ? 2 : 0)>{}, 2);

  f32x16 o0 = zero16(), o1 = zero16();
  const float sc = p.attn_scale * kLog2e;
  const int cb = 16 * ((lane >> 4) & 1);

  // one slot of work on ring buffer B; the copy for slot u + NB - 1 goes to the
  // buffer slot u - 1 used, which every wave has finished reading at the barrier
  auto step = [&](auto B, int u) __device__ {
    constexpr int b = decltype(B)::value;
    const int s = sSlot[u];
    wait_slots<L>(min(NB - 2, n - 1 - u));
    block_barrier();
    if (u + NB - 1 < n) issue(std::integral_constant<int, (b + NB - 1) % NB>{}, u + NB - 1);
    const T* sK = slot_buf(B);
    const T* sV = sK + TILE;
    // S^T (keys x queries): rows 0-31 in st0, 32-63 in st1
    f32x16 st0 = zero16(), st1 = zero16();
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const Frag<T> a0 = lds_frag(sK, lane & 31, 16 * kb + 8 * hh);
      const Frag<T> a1 = lds_frag(sK, 32 + (lane & 31), 16 * kb + 8 * hh);
      mma32(st0, a0, qf[kb]);
      mma32(st1, a1, qf[kb]);
    }

    // softmax of this lane's query over the chunk's 64 keys (base-2 domain)
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, fmaxf(st0[i], st1[i]));
    mx = fmaxf(mx, xor32(mx)) * sc;
    if (OBO) mx = fmaxf(mx, 0.f);
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      st0[i] = __builtin_amdgcn_exp2f(fmaf(st0[i], sc, -mx));
      st1[i] = __builtin_amdgcn_exp2f(fmaf(st1[i], sc, -mx));
      sum += st0[i] + st1[i];
    }
    sum += xor32(sum);
    if (OBO) sum += __builtin_amdgcn_exp2f(-mx);
    if (hh == 0) sLse[s * kS + qi] = (mx + __builtin_amdgcn_logf(sum)) * kLn2;

    // fuse w_s / l_s into P and accumulate O^T += V^T P^T
    const float coef = sW[s] / sum;
    Frag<T> pf[4];
    frag_from_acc(pf[0], st0, 0, coef);
    frag_from_acc(pf[1], st0, 1, coef);
    frag_from_acc(pf[2], st1, 0, coef);
    frag_from_acc(pf[3], st1, 1, coef);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const Frag<T> a0 = lds_frag_t(sV, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb);
      const Frag<T> a1 = lds_frag_t(sV, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb);
      mma32(o0, a0, pf[kb]);
      mma32(o1, a1, pf[kb]);
    }
  };
  for (int u0 = 0; u0 < n; u0 += NB) {
    step(std::integral_constant<int, 0>{}, u0);
    if (u0 + 1 < n) step(std::integral_constant<int, 1>{}, u0 + 1);
    if (NB > 2 && u0 + 2 < n) step(std::integral_constant<int, (NB > 2 ? 2 : 0)>{}, u0 + 2);
    if (NB > 3 && u0 + 3 < n) step(std::integral_constant<int, (NB > 3 ? 3 : 0)>{}, u0 + 3);
  }

  // O^T accumulator: lane holds query qi, d = 32*dt + 8*g + 4*hh + 0..3
  T* orow = out + qi * kD;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    store4(orow + 8 * g + 4 * hh, o0[4 * g], o0[4 * g + 1], o0[4 * g + 2], o0[4 * g + 3]);
    store4(orow + 32 + 8 * g + 4 * hh, o1[4 * g], o1[4 * g + 1], o1[4 * g + 2], o1[4 * g + 3]);
  }
  if (lse) {
    __syncthreads();
    for (int e = tid; e < kS * K; e += kThreads) {
      const int q = e / K, s = e % K;
      lse[e] = sJ[s] >= 0 ? sLse[s * kS + q] : -INFINITY;
    }
  }
}

}  // namespace

hipError_t launch_xattn_fwd(const Shape& s, const void* q, const void* k, const void* v,
                            const int32_t* idx, const float* sel, void* out, float* lse, float* w,
                            hipStream_t stream) {
  FwdParams p;
  p.q = q; p.k = k; p.v = v; p.idx = idx; p.sel = sel;
  p.out = out; p.lse = lse; p.w = w;
  p.H = s.H; p.Hr = s.Hr; p.topk = s.topk;
  p.nQ = s.nQ; p.nKV = s.nKV;
  p.nwork = (int64_t)s.B * s.H * s.nQ;
  p.causal = s.causal;
  p.attn_scale = s.attn_scale;
  const dim3 grid((unsigned)round8(p.nwork)), block(kThreads);
  if (s.bf16) {
    if (s.off_by_one) {
      hipLaunchKernelGGL((xattn_fwd_kernel<__bf16, true>), grid, block, 0, stream, p);
      note_launch("xattn_fwd_kernel", stream);
    }
    else {
      hipLaunchKernelGGL((xattn_fwd_kernel<__bf16, false>), grid, block, 0, stream, p);
      note_launch("xattn_fwd_kernel", stream);
    }
  } else {
    if (s.off_by_one) {
      hipLaunchKernelGGL((xattn_fwd_kernel<float, true>), grid, block, 0, stream, p);
      note_launch("xattn_fwd_kernel", stream);
    }
    else {
      hipLaunchKernelGGL((xattn_fwd_kernel<float, false>), grid, block, 0, stream, p);
      note_launch("xattn_fwd_kernel", stream);
    }
  }
  return take_launch_error();
}

}  // namespace gca
