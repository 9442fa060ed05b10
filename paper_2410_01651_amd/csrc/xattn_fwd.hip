// Grouped cross attention forward (Eq. 2-3 of the method; Algorithm 1 in the
// appendix is its tiled form).
//
// One workgroup of two waves per (batch, head, query chunk).  Each wave owns 32
// of the chunk's 64 query tokens and keeps their Q fragments in registers for
// the whole kernel.  For every retrieved chunk (slot) the workgroup gathers
// that chunk's 64 keys and values into LDS, computes S^T = K Q^T on the
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

template <typename T, bool OBO>
__global__ __launch_bounds__(kThreads) void xattn_fwd_kernel(FwdParams p) {
  constexpr int LD = LdsLd<T>::v;
  __shared__ __attribute__((aligned(16))) T sK[kS * LD];
  __shared__ __attribute__((aligned(16))) T sV[kS * LD];
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

  if (tid < 32) {
    float wv = 0.f;
    int jv = -1;
    if (t >= 0 && tid < K)
      row_weight(p.idx + (row_base + t) * K, p.sel + (row_base + t) * K, K, p.nKV, tid, wv, jv);
    sW[tid] = wv;
    sJ[tid] = jv;
    // every row's weights are written once: by the query chunk it feeds, and
    // the causal last row (which feeds no chunk) by chunk 0
    if (p.w && tid < K && (p.Hr != 1 || h == 0)) {
      const int64_t wt = p.causal ? (c == 0 ? p.nQ - 1 : c - 1) : 0;
      float ww;
      int jj;
      row_weight(p.idx + (row_base + wt) * K, p.sel + (row_base + wt) * K, K, p.nKV, tid, ww, jj);
      p.w[(row_base + wt) * K + tid] = ww;
    }
  }
  __syncthreads();
  if (tid == 0) {
    int n = 0;
    for (int s = 0; s < K; ++s)
      if (sJ[s] >= 0) sSlot[n++] = s;
    sN = n;
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

  const int64_t kv0 = (b * p.H + h) * p.nKV * (kS * kD);
  const T* kbase = reinterpret_cast<const T*>(p.k) + kv0;
  const T* vbase = reinterpret_cast<const T*>(p.v) + kv0;

  Tile64<T, kThreads> tk, tv;
  {
    const int64_t j0 = sJ[sSlot[0]];
    tk.load_cached(kbase + j0 * (kS * kD), tid);
    tv.load_cached(vbase + j0 * (kS * kD), tid);
  }
  f32x16 o0 = zero16(), o1 = zero16();
  const float sc = p.attn_scale * kLog2e;
  const int cb = 16 * ((lane >> 4) & 1);

  for (int u = 0; u < n; ++u) {
    const int s = sSlot[u];
    __syncthreads();
    tk.store(sK, LD, tid);
    tv.store(sV, LD, tid);
    __syncthreads();
    if (u + 1 < n) {
      const int64_t jn = sJ[sSlot[u + 1]];
      tk.load_cached(kbase + jn * (kS * kD), tid);
      tv.load_cached(vbase + jn * (kS * kD), tid);
    }

    // S^T (keys x queries): rows 0-31 in st0, 32-63 in st1
    f32x16 st0 = zero16(), st1 = zero16();
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const Frag<T> a0 = load_frag(sK + (lane & 31) * LD + 16 * kb + 8 * hh);
      const Frag<T> a1 = load_frag(sK + (32 + (lane & 31)) * LD + 16 * kb + 8 * hh);
      mma32(st0, a0, qf[kb]);
      mma32(st1, a1, qf[kb]);
    }

    // softmax of this lane's query over the chunk's 64 keys (base-2 domain)
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      st0[i] *= sc;
      st1[i] *= sc;
      mx = fmaxf(mx, fmaxf(st0[i], st1[i]));
    }
    mx = fmaxf(mx, xor32(mx));
    if (OBO) mx = fmaxf(mx, 0.f);
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      st0[i] = __builtin_amdgcn_exp2f(st0[i] - mx);
      st1[i] = __builtin_amdgcn_exp2f(st1[i] - mx);
      sum += st0[i] + st1[i];
    }
    sum += xor32(sum);
    if (OBO) sum += __builtin_amdgcn_exp2f(-mx);
    if (lse && hh == 0) lse[qi * K + s] = (mx + __builtin_amdgcn_logf(sum)) * kLn2;

    // fuse w_s / l_s into P and accumulate O^T += V^T P^T
    const float coef = sW[s] / sum;
    Frag<T> pf[4];
    frag_from_acc(pf[0], st0, 0, coef);
    frag_from_acc(pf[1], st0, 1, coef);
    frag_from_acc(pf[2], st1, 0, coef);
    frag_from_acc(pf[3], st1, 1, coef);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const Frag<T> a0 = load_frag_t(sV, LD, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb);
      const Frag<T> a1 = load_frag_t(sV, LD, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb);
      mma32(o0, a0, pf[kb]);
      mma32(o1, a1, pf[kb]);
    }
  }

  // O^T accumulator: lane holds query qi, d = 32*dt + 8*g + 4*hh + 0..3
  T* orow = out + qi * kD;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    store4(orow + 8 * g + 4 * hh, o0[4 * g], o0[4 * g + 1], o0[4 * g + 2], o0[4 * g + 3]);
    store4(orow + 32 + 8 * g + 4 * hh, o1[4 * g], o1[4 * g + 1], o1[4 * g + 2], o1[4 * g + 3]);
  }
  if (lse)
    for (int e = tid; e < kS * K; e += kThreads)
      if (sJ[e % K] < 0) lse[e] = -INFINITY;
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
