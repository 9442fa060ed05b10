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

// Per-lane retrieval metadata of one landmark row: lane s < K holds slot s's
// chunk index and raw score (chunk -1 for lanes >= K or rows that do not exist).
struct RowMeta {
  int j;
  float sv;
};

// Position (b, h, c) of work item w = (b * H + h) * nQ + c, stepped one chunk at a
// time so the persistent loop needs no divisions.
struct Geo {
  int64_t b, c;
  int h;
  __device__ __forceinline__ Geo(int64_t w, int64_t nQ, int H) {
    c = w % nQ;
    const int64_t bh = w / nQ;
    h = (int)(bh % H);
    b = bh / H;
  }
  __device__ __forceinline__ void next(int64_t nQ, int H, int64_t step) {
    c += step;
    while (c >= nQ) {
      c -= nQ;
      if (++h == H) {
        h = 0;
        ++b;
      }
    }
  }
};

__device__ __forceinline__ RowMeta load_row_meta(const FwdParams& p, int64_t row_off, bool exists) {
  const int lane = threadIdx.x & 63;
  RowMeta m{-1, -INFINITY};
  if (exists && lane < p.topk) {
    m.j = p.idx[row_off + lane];
    m.sv = p.sel[row_off + lane];
  }
  return m;
}

template <typename T, bool OBO>
__global__ __launch_bounds__(kThreads, 2) void xattn_fwd_kernel(FwdParams p) {
  constexpr int TILE = kS * kD;
  __shared__ __attribute__((aligned(16))) T ring[4 * 2 * TILE];  // 4 slots: a chunk's K and V tiles
  __shared__ float sLse[32 * kS];  // current chunk: [slot][query]
  __shared__ int sJ[2][32];        // per slot: chunk index or -1 (current and next chunk)
  __shared__ int sSlot[2][32];     // compacted lists of valid slots: slot, chunk, weight
  __shared__ int sJc[2][32];
  __shared__ float sWc[2][32];
  __shared__ int sN[2];

  // Work order: workgroups are dealt to the eight XCDs round-robin (blockIdx mod
  // 8).  XCD x owns the x-th eighth of the chunks, and its workgroups sweep that
  // range side by side (workgroup k takes chunks begin + k, + k + G, ...; G = its
  // XCD's workgroup count), so at any time each XCD works on a window of
  // consecutive query chunks of one (batch, head) slice.  The retrieved key and
  // value chunks then come from a few slices at a time, which the XCD's L2 and
  // the shared last-level cache keep resident across the queries that reuse them.
  const int64_t stride = gridDim.x >> 3;
  const int xcd = (int)(blockIdx.x & 7);
  const int64_t c_begin = p.nwork * xcd / 8 + (blockIdx.x >> 3);
  const int64_t c_end = p.nwork * (xcd + 1) / 8;
  if (c_begin >= c_end) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5;
  const int pair = wave >> 1, half = wave & 1;
  const int K = p.topk;
  const int qi = 32 * half + (lane & 31);  // this lane's query token within a chunk
  const float sc = p.attn_scale * kLog2e;
  const int cb = 16 * ((lane >> 4) & 1);

  // work item w = (b, h, c): geometry helpers
  auto row_of = [&](const Geo& g, int64_t& row_off, bool& exists, bool& owner) __device__ {
    const int hr = p.Hr == 1 ? 0 : g.h;
    const int64_t t = p.causal ? g.c - 1 : 0;
    exists = t >= 0;
    row_off = ((g.b * p.Hr + hr) * p.nQ + (exists ? t : 0)) * K;
    owner = p.Hr != 1 || g.h == 0;  // writes the row's weights
  };
  // wave 0: turn a row's metadata into the compacted slot list of buffer par
  auto make_slots = [&](const RowMeta& m, const Geo& g, int par) __device__ {
    int64_t row_off;
    bool exists, owner;
    row_of(g, row_off, exists, owner);
    const bool valid = lane < K && m.j >= 0 && m.j < p.nKV;
    float mx = valid ? m.sv : -INFINITY;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    const float e = valid ? expf(m.sv - mx) : 0.f;
    float sum = e;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o);
    const float wv = valid ? e / sum : 0.f;
    const uint64_t mask = __ballot(valid);
    if (lane < 32) sJ[par][lane] = valid ? m.j : -1;
    if (valid) {
      const int rk = __popcll(mask & ((1ull << lane) - 1));
      sSlot[par][rk] = lane;
      sJc[par][rk] = m.j;
      sWc[par][rk] = wv;
    }
    if (lane == 0) sN[par] = __popcll(mask);
    if (p.w && exists && owner && lane < K) p.w[row_off + lane] = wv;
  };
  auto qrow_ptr = [&](int64_t w) __device__ {
    return reinterpret_cast<const T*>(p.q) + (w * kS + qi) * kD;
  };

  // ---- prologue: the first chunk's slot list and Q, the second chunk's metadata
  Frag<T> qf[4], qn[4];
  RowMeta meta{-1, -INFINITY};
  Geo g0(c_begin, p.nQ, p.H);  // geometry of the current chunk and of the two after it
  Geo g1 = g0;
  g1.next(p.nQ, p.H, stride);
  Geo g2 = g1;
  g2.next(p.nQ, p.H, stride);
  {
    int64_t ro;
    bool ex, ow;
    row_of(g0, ro, ex, ow);
    const RowMeta m0 = load_row_meta(p, ro, ex);
    const T* qr = qrow_ptr(c_begin);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) qf[kb] = load_frag(qr + 16 * kb + 8 * hh);
    if (wave == 0) make_slots(m0, g0, 0);
    if (c_begin + stride < c_end) {
      row_of(g1, ro, ex, ow);
      meta = load_row_meta(p, ro, ex);
    }
    wait_vmem<0>();
    __syncthreads();
  }

  // the ring: global round counter picks the slot pair (rounds alternate slots 0,1 / 2,3)
  int round = 0;
  const TileCopy<T, 4> cp(wave, lane);
  const T* const gk = reinterpret_cast<const T*>(p.k);
  const T* const gv = reinterpret_cast<const T*>(p.v);
  // element offset of the (batch, head) key/value slice of chunk w
  auto slice_of = [&](const Geo& g) __device__ { return (g.b * p.H + g.h) * p.nKV * TILE; };
  auto issue_item = [&](int64_t kvb, int j, int slot) __device__ {
    T* dst = ring + slot * (2 * TILE);
    cp.issue(gk + kvb + (int64_t)j * TILE, dst);
    cp.issue(gv + kvb + (int64_t)j * TILE, dst + TILE);
  };
  // lane u < 32 of each list holds valid item u of the current chunk (slot, chunk,
  // weight) or of the next chunk (chunk); items are picked with a lane read
  const int l32 = lane & 31;
  int ls = sSlot[0][l32], lj = sJc[0][l32], ljn = 0;
  float lw = sWc[0][l32];
  int64_t kvb = slice_of(g0), kvb_n = 0;
  // copies of round 0 of the first chunk
  if (sN[0] > 0) issue_item(kvb, __builtin_amdgcn_readlane(lj, 0), 0);
  if (sN[0] > 1) issue_item(kvb, __builtin_amdgcn_readlane(lj, 1), 1);

  auto compute = [&](const T* sK, int u, f32x16& o0, f32x16& o1) __device__ {
    const int s = __builtin_amdgcn_readlane(ls, u);
    const T* sV = sK + TILE;
    // all K fragments first, so the eight products issue back to back
    Frag<T> ka[8];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      ka[2 * kb] = lds_frag(sK, lane & 31, 16 * kb + 8 * hh);
      ka[2 * kb + 1] = lds_frag(sK, 32 + (lane & 31), 16 * kb + 8 * hh);
    }
    f32x16 st0 = zero16(), st1 = zero16();
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      mma32(st0, ka[2 * kb], qf[kb]);
      mma32(st1, ka[2 * kb + 1], qf[kb]);
    }
    // V^T fragments are read while the softmax runs
    Frag<T> va[8];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      va[2 * kb] = lds_frag_t(sV, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb);
      va[2 * kb + 1] = lds_frag_t(sV, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, fmaxf(st0[i], st1[i]));
    mx = max_xor32(mx) * sc;
    if (OBO) mx = fmaxf(mx, 0.f);
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      st0[i] = __builtin_amdgcn_exp2f(fmaf(st0[i], sc, -mx));
      st1[i] = __builtin_amdgcn_exp2f(fmaf(st1[i], sc, -mx));
      sum += st0[i] + st1[i];
    }
    sum = sum_xor32(sum);
    if (OBO) sum += __builtin_amdgcn_exp2f(-mx);
    if (hh == 0) sLse[s * kS + qi] = (mx + __builtin_amdgcn_logf(sum)) * kLn2;
    const int coef_bits = __builtin_amdgcn_readlane(__float_as_int(lw), u);
    const float coef = __int_as_float(coef_bits) * __builtin_amdgcn_rcpf(sum);
    Frag<T> pf[4];
    frag_from_acc(pf[0], st0, 0, coef);
    frag_from_acc(pf[1], st0, 1, coef);
    frag_from_acc(pf[2], st1, 0, coef);
    frag_from_acc(pf[3], st1, 1, coef);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      mma32(o0, va[2 * kb], pf[kb]);
      mma32(o1, va[2 * kb + 1], pf[kb]);
    }
  };

  int par = 0;
  for (int64_t w = c_begin; w < c_end; w += stride, par ^= 1) {
    const int n = sN[par];
    const int R = n > 0 ? (n + 1) / 2 : 1;
    const bool has_next = w + stride < c_end;
    f32x16 o0 = zero16(), o1 = zero16();
    for (int r = 0; r < R; ++r) {
      wait_vmem<0>();
      block_barrier();
      if (r == 0) {
        if (w != c_begin) {
#pragma unroll
          for (int kb = 0; kb < 4; ++kb) qf[kb] = qn[kb];
          ls = sSlot[par][l32];
          lj = sJc[par][l32];
          lw = sWc[par][l32];
          kvb = kvb_n;
        }
        if (has_next) {
          const T* qr = qrow_ptr(w + stride);
#pragma unroll
          for (int kb = 0; kb < 4; ++kb) qn[kb] = load_frag(qr + 16 * kb + 8 * hh);
          if (wave == 0) make_slots(meta, g1, par ^ 1);
          if (w + 2 * stride < c_end) {
            int64_t ro;
            bool ex, ow;
            row_of(g2, ro, ex, ow);
            meta = load_row_meta(p, ro, ex);
          }
        }
        block_barrier();  // the next chunk's slot list is visible
        if (has_next) {
          ljn = sJc[par ^ 1][l32];
          kvb_n = slice_of(g1);
        }
      }
      const int cur = 2 * (round & 1), nxt = 2 - cur;
      if (r + 1 < R) {
        if (2 * r + 2 < n) issue_item(kvb, __builtin_amdgcn_readlane(lj, 2 * r + 2), nxt);
        if (2 * r + 3 < n) issue_item(kvb, __builtin_amdgcn_readlane(lj, 2 * r + 3), nxt + 1);
      } else if (has_next) {
        const int nn = sN[par ^ 1];
        if (nn > 0) issue_item(kvb_n, __builtin_amdgcn_readlane(ljn, 0), nxt);
        if (nn > 1) issue_item(kvb_n, __builtin_amdgcn_readlane(ljn, 1), nxt + 1);
      }
      const int u = 2 * r + pair;
      if (u < n) compute(ring + (cur + pair) * (2 * TILE), u, o0, o1);
      ++round;
    }

    // ---- finish chunk w: pair 1 hands its partial O^T to pair 0 through this
    // round's ring slot, which no copy targets until the next round's barrier
    const int64_t tok0 = w * kS;
    T* out = reinterpret_cast<T*>(p.out) + tok0 * kD;
    float* part = reinterpret_cast<float*>(ring + (((round - 1) & 1) == 0 ? 1 : 3) * (2 * TILE));
    block_barrier();
    if (pair == 1 && n > 1) {
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        *reinterpret_cast<f32x4*>(part + ((half * 4 + gq) * 2 + 0) * 256 + lane * 4) =
            f32x4{o0[4 * gq], o0[4 * gq + 1], o0[4 * gq + 2], o0[4 * gq + 3]};
        *reinterpret_cast<f32x4*>(part + ((half * 4 + gq) * 2 + 1) * 256 + lane * 4) =
            f32x4{o1[4 * gq], o1[4 * gq + 1], o1[4 * gq + 2], o1[4 * gq + 3]};
      }
    }
    block_barrier();
    if (pair == 0) {
      T* orow = out + qi * kD;
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        f32x4 a{0.f, 0.f, 0.f, 0.f}, bq{0.f, 0.f, 0.f, 0.f};
        if (n > 1) {
          a = *reinterpret_cast<const f32x4*>(part + ((half * 4 + gq) * 2 + 0) * 256 + lane * 4);
          bq = *reinterpret_cast<const f32x4*>(part + ((half * 4 + gq) * 2 + 1) * 256 + lane * 4);
        }
        store4(orow + 8 * gq + 4 * hh, o0[4 * gq] + a[0], o0[4 * gq + 1] + a[1], o0[4 * gq + 2] + a[2],
               o0[4 * gq + 3] + a[3]);
        store4(orow + 32 + 8 * gq + 4 * hh, o1[4 * gq] + bq[0], o1[4 * gq + 1] + bq[1], o1[4 * gq + 2] + bq[2],
               o1[4 * gq + 3] + bq[3]);
      }
    }
    if (p.lse) {
      float* lse = p.lse + (tok0 + lane) * K;
      for (int s = wave; s < K; s += 4) lse[s] = sJ[par][s] >= 0 ? sLse[s * kS + lane] : -INFINITY;
    }
    // the causal last row feeds no chunk: its weights go out with chunk 0
    if (p.w && p.causal && g0.c == 0 && wave == 1) {
      int64_t ro;
      bool ex, ow;
      row_of(g0, ro, ex, ow);
      if (ow) {
        const int64_t last_off = (g0.b * p.Hr + (p.Hr == 1 ? 0 : g0.h)) * p.nQ * K + (p.nQ - 1) * K;
        float wv;
        int jv;
        wave_row_weight(p.idx, p.sel, last_off, K, p.nKV, wv, jv);
        if (lane < K) p.w[last_off + lane] = wv;
      }
    }
    g0 = g1;
    g1 = g2;
    g2.next(p.nQ, p.H, stride);
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
  // persistent workgroups: two per CU (256 CUs), a multiple of 8 (one share per XCD)
  const int64_t target = 512;
  const dim3 grid((unsigned)(p.nwork < target ? round8(p.nwork) : target)), block(kThreads);
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
