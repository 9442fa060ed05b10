// Grouped cross attention forward (Eq. 2-3 of the method; Algorithm 1 in the
// appendix is its tiled form).
//
// One workgroup of four waves per (batch, head, query chunk): two pairs of
// waves take alternate retrieved chunks, and within a pair each wave owns 32 of
// the chunk's 64 query tokens and keeps their Q fragments in registers.  The
// retrieved chunks' keys and values stream through a four-slot LDS ring filled
// by asynchronous direct-to-LDS copies one round ahead of the compute (two
// waves per SIMD hide each other's MFMA, LDS and cross-lane latencies).  For
// every retrieved chunk (slot) a pair computes S^T = K Q^T on the
// matrix cores, takes each query's softmax over the 64 keys (one retrieved
// chunk is exactly one tile, so no running rescale is needed), folds the
// fusion weight w_s / l_s into P, and accumulates O^T += V^T (w_s P_s)^T into one
// fp32 accumulator per pair; the two pairs' accumulators are summed at the end.  The per-chunk outputs O'_s of
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

constexpr int kThreads = 256;  // two pairs of waves

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

template <typename T, bool OBO>
__global__ __launch_bounds__(kThreads) void xattn_fwd_kernel(FwdParams p) {
  constexpr int TILE = kS * kD;
  GCA_RING4(T, 2 * TILE)           // each slot: one retrieved chunk's K and V tiles
  __shared__ float sLse[32 * kS];  // [slot][query]
  __shared__ float sW[32];
  __shared__ int sJ[32];
  __shared__ int sSlot[32];
  __shared__ int sN;

  const int64_t wid = xcd_swizzle(blockIdx.x, gridDim.x);
  if (wid >= p.nwork) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5;
  const int pair = wave >> 1, half = wave & 1;
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
  if (wave == 0 || (wave == 1 && p.w && p.causal && c == 0 && (p.Hr != 1 || h == 0))) {
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

  const int qi = 32 * half + (lane & 31);  // this lane's query token within the chunk
  const T* qrow = reinterpret_cast<const T*>(p.q) + (tok0 + qi) * kD;
  Frag<T> qf[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) qf[kb] = load_frag(qrow + 16 * kb + 8 * hh);
  wait_vmem<0>();  // nothing but the chunk copies may be pending inside the slot loop

  const int64_t kv0 = (b * p.H + h) * p.nKV * TILE;
  const T* kbase = reinterpret_cast<const T*>(p.k) + kv0;
  const T* vbase = reinterpret_cast<const T*>(p.v) + kv0;
  auto issue = [&](auto B, int u) __device__ {
    const int64_t j = sJ[sSlot[u]];
    T* dst = slot_buf(B);
    dma_tile<T, 4>(kbase + j * TILE, dst, wave, lane);
    dma_tile<T, 4>(vbase + j * TILE, dst + TILE, wave, lane);
  };

  f32x16 o0 = zero16(), o1 = zero16();
  const float sc = p.attn_scale * kLog2e;
  const int cb = 16 * ((lane >> 4) & 1);

  auto run = [&](auto B, int u) __device__ {
    const int s = sSlot[u];
    const T* sK = slot_buf(B);
    const T* sV = sK + TILE;
    // S^T (keys x queries): rows 0-31 in st0, 32-63 in st1
    f32x16 st0 = zero16(), st1 = zero16();
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      mma32(st0, lds_frag(sK, lane & 31, 16 * kb + 8 * hh), qf[kb]);
      mma32(st1, lds_frag(sK, 32 + (lane & 31), 16 * kb + 8 * hh), qf[kb]);
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
      mma32(o0, lds_frag_t(sV, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb), pf[kb]);
      mma32(o1, lds_frag_t(sV, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb), pf[kb]);
    }
  };
  pair_ring(n, pair, issue, run);

  // pair 1 hands its partial O^T to pair 0 through LDS (the ring is free now)
  float* part = reinterpret_cast<float*>(ring0);  // [query][d] fp32, 16 KB
  __syncthreads();
  if (pair == 1) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      *reinterpret_cast<f32x4*>(part + qi * kD + 8 * g + 4 * hh) =
          f32x4{o0[4 * g], o0[4 * g + 1], o0[4 * g + 2], o0[4 * g + 3]};
      *reinterpret_cast<f32x4*>(part + qi * kD + 32 + 8 * g + 4 * hh) =
          f32x4{o1[4 * g], o1[4 * g + 1], o1[4 * g + 2], o1[4 * g + 3]};
    }
  }
  __syncthreads();
  if (pair == 0) {
    // O^T accumulator: lane holds query qi, d = 32*dt + 8*g + 4*hh + 0..3
    T* orow = out + qi * kD;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 a = *reinterpret_cast<const f32x4*>(part + qi * kD + 8 * g + 4 * hh);
      const f32x4 bq = *reinterpret_cast<const f32x4*>(part + qi * kD + 32 + 8 * g + 4 * hh);
      store4(orow + 8 * g + 4 * hh, o0[4 * g] + a[0], o0[4 * g + 1] + a[1], o0[4 * g + 2] + a[2],
             o0[4 * g + 3] + a[3]);
      store4(orow + 32 + 8 * g + 4 * hh, o1[4 * g] + bq[0], o1[4 * g + 1] + bq[1], o1[4 * g + 2] + bq[2],
             o1[4 * g + 3] + bq[3]);
    }
  }
  if (lse) {
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
