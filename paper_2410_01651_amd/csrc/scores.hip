// Causal relevance scores and top-k retrieval (Eq. 1 of the method).
//
// chunk_scores: the landmark score matrix r[t, j] = scale * <lmk_q[t], lmk_k[j]>
//   as 64x64 output tiles on the matrix cores (each wave one 32x32 block),
//   with the strictly-upper causal region filled with -inf and fully masked
//   tiles skipping the product.
// topk: one wave per score row; every lane keeps a sorted best-KM list of the
//   columns it visits, and the 64 lists are merged k times with a wave-wide
//   lexicographic (score desc, chunk asc) reduction.  The chosen chunks are
//   then written in ascending chunk order.
// decode select: one landmark query against every past landmark key.  The
//   keys are read once, coalesced, by many workgroups that each own a slice;
//   8 lanes share one key row (16 bytes each per step) and reduce the dot
//   product with two cross-lane steps.  Each workgroup leaves its slice's best
//   k in the workspace and one workgroup per row merges them.
#include "gca_device.hpp"
#include "gca_launch.hpp"

namespace gca {
namespace {

// ------------------------------------------------------------ scores ----

template <typename T>
__global__ __launch_bounds__(256) void chunk_scores_kernel(const T* __restrict__ lq, const T* __restrict__ lk,
                                                           float* __restrict__ scores, int64_t nQ, int64_t nC,
                                                           int D, float scale, int causal, int64_t ntq,
                                                           int64_t ntj, int64_t nwork) {
  const int64_t wid = xcd_swizzle(blockIdx.x, gridDim.x);
  if (wid >= nwork) return;
  const int64_t tj = wid % ntj;
  const int64_t rest = wid / ntj;
  const int64_t tq = rest % ntq;
  const int64_t bhr = rest / ntq;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
  const int64_t t0 = tq * 64 + 32 * (wave >> 1);
  const int64_t j0 = tj * 64 + 32 * (wave & 1);
  const int64_t j = j0 + (lane & 31);
  float* out = scores + bhr * nQ * nC;

  f32x16 acc = zero16();
  const bool any = !causal || (j0 < t0 + 31);  // some j < t inside this 32x32 block
  if (any && t0 < nQ && j0 < nC) {
    const int64_t ta = t0 + (lane & 31) < nQ ? t0 + (lane & 31) : nQ - 1;  // clamped rows are discarded
    const int64_t jb = j < nC ? j : nC - 1;
    const T* arow = lq + (bhr * nQ + ta) * D;
    const T* brow = lk + (bhr * nC + jb) * D;
    for (int x = 0; x < D; x += 16) {
      const Frag<T> a = load_frag(arow + x + 8 * hh);
      const Frag<T> bb = load_frag(brow + x + 8 * hh);
      mma32(acc, a, bb);
    }
  }
  if (j < nC) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t t = t0 + 8 * (i >> 2) + 4 * hh + (i & 3);
      if (t < nQ) out[t * nC + j] = (!causal || j < t) ? acc[i] * scale : -INFINITY;
    }
  }
}

// ------------------------------------------------------------- top-k ----

template <int KM>
__device__ __forceinline__ void write_sorted(int32_t* idx, float* sel, int K, float ms, int mj, int cnt) {
  const int lane = threadIdx.x & 63;
  const int rank = rank_by_chunk(mj, cnt);
  if (lane < cnt) {
    idx[rank] = mj;
    sel[rank] = ms;
  } else if (lane < K) {
    idx[lane] = -1;
    sel[lane] = -INFINITY;
  }
}

template <int KM>
__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ scores, int32_t* __restrict__ idx,
                                                   float* __restrict__ sel, int64_t rows, int64_t nQ,
                                                   int64_t nC, int K, int causal) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t t = row % nQ;
  const int64_t lim = causal ? (t < nC ? t : nC) : nC;
  const float* sr = scores + row * nC;
  TopList<KM> L;
  L.init();
  for (int64_t j = lane; j < lim; j += 64) {
    const float v = sr[j];
    if (__builtin_isfinite(v)) L.insert(v, (int)j);
  }
  float ms;
  int mj, cnt;
  wave_merge(L, K, ms, mj, cnt);
  write_sorted<KM>(idx + row * K, sel + row * K, K, ms, mj, cnt);
}

// ------------------------------------------------------- decode select ----

constexpr int kScanThreads = 256;
constexpr int kMaxScanSlices = 1024;

struct ScanPlan {
  int64_t per;     // keys per slice
  int64_t slices;  // slices per retrieval row
};

// 8-element dot product accumulated in fp32 (bf16 products are exact in fp32).
__device__ __forceinline__ float dot8(const bf16x8& a, const bf16x8& b, float acc) {
#pragma unroll
  for (int m = 0; m < 8; ++m) acc = fmaf((float)a[m], (float)b[m], acc);
  return acc;
}
__device__ __forceinline__ float dot8(const f32x8& a, const f32x8& b, float acc) {
  acc = fmaf(a.lo[0], b.lo[0], acc); acc = fmaf(a.lo[1], b.lo[1], acc);
  acc = fmaf(a.lo[2], b.lo[2], acc); acc = fmaf(a.lo[3], b.lo[3], acc);
  acc = fmaf(a.hi[0], b.hi[0], acc); acc = fmaf(a.hi[1], b.hi[1], acc);
  acc = fmaf(a.hi[2], b.hi[2], acc); acc = fmaf(a.hi[3], b.hi[3], acc);
  return acc;
}

ScanPlan scan_plan(int64_t nC) {
  int64_t per = (nC + kMaxScanSlices - 1) / kMaxScanSlices;
  if (per < 256) per = 256;
  per = (per + 31) & ~int64_t(31);
  ScanPlan p;
  p.per = per;
  p.slices = (nC + per - 1) / per;
  return p;
}

// Wave-level merge, then merge of the workgroup's NW wave results by wave 0.
// Leaves the workgroup's best (<= K) in lanes of wave 0: (ms, mj), cnt.
// sS/sJ hold NW * 32 entries, sCnt NW.
template <int KM, int NW>
__device__ __forceinline__ void block_merge(TopList<KM>& L, int K, float* sS, int* sJ, int* sCnt, float& ms,
                                            int& mj, int& cnt) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  wave_merge(L, K, ms, mj, cnt);
  if (lane < 32) {
    sS[wave * 32 + lane] = ms;
    sJ[wave * 32 + lane] = mj;
  }
  if (lane == 0) sCnt[wave] = cnt;
  __syncthreads();
  if (wave == 0) {
    L.init();
#pragma unroll
    for (int w0 = 0; w0 < NW; w0 += 2) {
      const int w = w0 + (lane >> 5);  // lanes 0-31 take wave w0, lanes 32-63 wave w0 + 1
      if (w < NW && (lane & 31) < sCnt[w]) L.insert(sS[w * 32 + (lane & 31)], sJ[w * 32 + (lane & 31)]);
    }
    wave_merge(L, K, ms, mj, cnt);
  }
}

template <typename T, int KM>
__global__ __launch_bounds__(kScanThreads) void decode_scan_kernel(const T* __restrict__ lq,
                                                                   const T* __restrict__ lk, float* __restrict__ cs,
                                                                   int* __restrict__ cj, int64_t nC, int D,
                                                                   float scale, int K, int64_t per,
                                                                   int64_t slices) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  T* sq = reinterpret_cast<T*>(smem);
  __shared__ float sS[kScanThreads / 64 * 32];
  __shared__ int sJ[kScanThreads / 64 * 32];
  __shared__ int sCnt[kScanThreads / 64];

  const int64_t g = blockIdx.x % slices;
  const int64_t bhr = blockIdx.x / slices;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, sub = lane & 7;
  const T* q = lq + bhr * D;  // the one landmark query of this row
  for (int x = tid * (16 / (int)sizeof(T)); x < D; x += kScanThreads * (16 / (int)sizeof(T)))
    *reinterpret_cast<u32x4*>(sq + x) = *reinterpret_cast<const u32x4*>(q + x);
  __syncthreads();

  const int64_t lo = g * per;
  const int64_t hi = lo + per < nC ? lo + per : nC;
  TopList<KM> L;
  L.init();
  // a wave scores two groups of 8 keys per round (lane: key lane/8, 16-byte
  // column block lane%8 of every 128 bytes), so 2 * D/64 loads are in flight
  constexpr int kWaves = kScanThreads / 64;
  int it = 0;
  for (int64_t base = lo + wave * 16; base < hi; base += 16 * kWaves, it += 2) {
    const int64_t key0 = base + (lane >> 3), key1 = key0 + 8;
    const T* kr0 = lk + (bhr * nC + (key0 < hi ? key0 : lo)) * D;
    const T* kr1 = lk + (bhr * nC + (key1 < hi ? key1 : lo)) * D;
    float acc0 = 0.f, acc1 = 0.f;
#pragma unroll 4
    for (int x = sub * 8; x < D; x += 64) {
      const Frag<T> a0 = load_frag(kr0 + x);
      const Frag<T> a1 = load_frag(kr1 + x);
      const Frag<T> b = load_frag(sq + x);
      acc0 = dot8(a0, b, acc0);
      acc1 = dot8(a1, b, acc1);
    }
    // sum over the key's 8 lanes (lanes 8m .. 8m+7: quad swaps, then the other quad)
    acc0 += dpp<kDppXor1>(acc0);
    acc1 += dpp<kDppXor1>(acc1);
    acc0 += dpp<kDppXor2>(acc0);
    acc1 += dpp<kDppXor2>(acc1);
    acc0 += dpp<kDppHalfMirror>(acc0);
    acc1 += dpp<kDppHalfMirror>(acc1);
    // spread the insertions of one key group over its 8 lanes
    if (key0 < hi && sub == (it & 7)) {
      const float v = acc0 * scale;
      if (__builtin_isfinite(v)) L.insert(v, (int)key0);
    }
    if (key1 < hi && sub == ((it + 1) & 7)) {
      const float v = acc1 * scale;
      if (__builtin_isfinite(v)) L.insert(v, (int)key1);
    }
  }
  float ms;
  int mj, cnt;
  block_merge<KM, kScanThreads / 64>(L, K, sS, sJ, sCnt, ms, mj, cnt);
  if (wave == 0 && lane < K) {
    const int64_t o = (bhr * slices + g) * K + lane;
    cs[o] = lane < cnt ? ms : -INFINITY;
    cj[o] = lane < cnt ? mj : -1;
  }
}

constexpr int kMergeThreads = 1024;

// Final top-k of one row from the slices' lists (each sorted best first).  The
// k-th best slice maximum T is a lower bound for the row's k-th best, so only
// candidates at or above T can win, and they come from the k slices whose
// maximum is at or above T: at most k * k candidates.  One pass finds T from
// the slice maxima, one pass gathers the candidates into LDS, one wave merges
// them.
template <int KM>
__global__ __launch_bounds__(kMergeThreads) void decode_merge_kernel(const float* __restrict__ cs,
                                                                     const int* __restrict__ cj,
                                                                     int32_t* __restrict__ idx,
                                                                     float* __restrict__ sel, int K,
                                                                     int64_t slices) {
  constexpr int NW = kMergeThreads / 64;
  constexpr int kMaxCand = 32 * 32;
  __shared__ float sS[NW * 32];
  __shared__ int sJ[NW * 32];
  __shared__ int sCnt[NW];
  __shared__ float sCs[kMaxCand];
  __shared__ int sCj[kMaxCand];
  __shared__ int sNc;
  __shared__ float sTs;
  __shared__ int sTj;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bhr = blockIdx.x;
  const int64_t n = slices * K;
  const float* c_s = cs + bhr * n;
  const int* c_j = cj + bhr * n;

  // 1. the threshold: k-th best of the slice maxima (slices <= kMergeThreads)
  TopList<KM> L;
  L.init();
  if (tid < slices) {
    const int j = c_j[(int64_t)tid * K];
    if (j >= 0) L.insert(c_s[(int64_t)tid * K], j);
  }
  float ms;
  int mj, cnt;
  block_merge<KM, NW>(L, K, sS, sJ, sCnt, ms, mj, cnt);
  if (wave == 0) {
    const float ts = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ms), K - 1));
    const int tj = __builtin_amdgcn_readlane(mj, K - 1);
    if (lane == 0) {
      sTs = cnt >= K ? ts : -INFINITY;  // fewer than k maxima: every candidate qualifies
      sTj = cnt >= K ? tj : kNoChunk;
      sNc = 0;
    }
  }
  __syncthreads();

  // 2. gather the candidates at or above the threshold
  const float ts = sTs;
  const int tj = sTj;
  for (int64_t e = tid; e < n; e += kMergeThreads) {
    const int j = c_j[e];
    if (j < 0) continue;
    const float v = c_s[e];
    if (!better(ts, tj, v, j)) {
      const int pos = atomicAdd(&sNc, 1);
      if (pos < kMaxCand) {
        sCs[pos] = v;
        sCj[pos] = j;
      }
    }
  }
  __syncthreads();

  // 3. one wave merges them
  if (wave == 0) {
    const int nc = min(sNc, kMaxCand);
    L.init();
    for (int i = lane; i < nc; i += 64) L.insert(sCs[i], sCj[i]);
    wave_merge(L, K, ms, mj, cnt);
    write_sorted<KM>(idx + bhr * K, sel + bhr * K, K, ms, mj, cnt);
  }
}

// ------------------------------------------------ fused causal select ----

// Scores and top-k in one pass for a block of 64 landmark rows: the workgroup
// walks the key tiles j < t in order, computes each 64x64 score tile on the
// matrix cores into LDS, and 4 threads per row fold the tile into their
// running best-KM lists.  No score matrix is written.  Row blocks are issued
// longest first (block tq has tq+1 tiles) so the triangular work balances.
template <typename T, int KM>
__global__ __launch_bounds__(256) void fused_select_kernel(const T* __restrict__ lq, const T* __restrict__ lk,
                                                           int32_t* __restrict__ idx, float* __restrict__ sel,
                                                           int64_t nQ, int64_t nC, int D, float scale, int K,
                                                           int64_t ntq) {
  __shared__ float sT[64][65];
  __shared__ float sRs[64][32];
  __shared__ int sRj[64][32];
  __shared__ int sCnt[64];
  const int64_t bhr = blockIdx.x / ntq;
  const int64_t tq = ntq - 1 - blockIdx.x % ntq;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5;
  const int r = tid >> 2, u = tid & 3;  // top-k duty: row r of the block, columns u, u+4, ...
  const int64_t t0 = tq * 64;
  const int64_t jend = t0 + 63 < nC ? t0 + 63 : nC;  // columns j < t <= t0 + 63
  TopList<KM> L;
  L.init();
  const int64_t rt0 = t0 + 32 * (wave >> 1);
  for (int64_t j0 = 0; j0 < jend; j0 += 64) {
    const int64_t cj0 = j0 + 32 * (wave & 1);
    const bool any = rt0 < nQ && cj0 < nC && cj0 < rt0 + 31;
    f32x16 acc = zero16();
    if (any) {
      const int64_t ta = rt0 + (lane & 31) < nQ ? rt0 + (lane & 31) : nQ - 1;
      const int64_t jb = cj0 + (lane & 31) < nC ? cj0 + (lane & 31) : nC - 1;
      const T* arow = lq + (bhr * nQ + ta) * D;
      const T* brow = lk + (bhr * nC + jb) * D;
      for (int x = 0; x < D; x += 16) {
        const Frag<T> a = load_frag(arow + x + 8 * hh);
        const Frag<T> bb = load_frag(brow + x + 8 * hh);
        mma32(acc, a, bb);
      }
    }
    const int jl = 32 * (wave & 1) + (lane & 31);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int tl = 32 * (wave >> 1) + 8 * (i >> 2) + 4 * hh + (i & 3);
      const int64_t t = t0 + tl, j = j0 + jl;
      sT[tl][jl] = (any && t < nQ && j < nC && j < t) ? acc[i] * scale : -INFINITY;
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const int c = u + 4 * m;
      const float v = sT[r][c];
      if (__builtin_isfinite(v)) L.insert(v, (int)(j0 + c));
    }
    __syncthreads();
  }
  // merge the row's 4 lists (lanes 4r .. 4r+3 of one wave)
  int cnt = 0;
  for (int s = 0; s < K; ++s) {
    float bs = L.s[0];
    int bj = L.j[0];
    take_better(bs, bj, dpp<kDppXor1>(bs), dpp<kDppXor1>(bj));
    take_better(bs, bj, dpp<kDppXor2>(bs), dpp<kDppXor2>(bj));
    if (bj != kNoChunk) {
      if (L.j[0] == bj) L.pop();
      if (u == 0) { sRs[r][cnt] = bs; sRj[r][cnt] = bj; }
      ++cnt;
    }
  }
  if (u == 0) sCnt[r] = cnt;
  __syncthreads();
  const int64_t t = t0 + r;
  if (t < nQ) {
    const int n = sCnt[r];
    int32_t* io = idx + (bhr * nQ + t) * K;
    float* so = sel + (bhr * nQ + t) * K;
    for (int e = u; e < K; e += 4) {
      if (e < n) {
        const int je = sRj[r][e];
        int rank = 0;
        for (int e2 = 0; e2 < n; ++e2) rank += sRj[r][e2] < je ? 1 : 0;
        io[rank] = je;
        so[rank] = sRs[r][e];
      } else {
        io[e] = -1;
        so[e] = -INFINITY;
      }
    }
  }
}

template <typename T, int KM>
hipError_t launch_fused_k(const Shape& s, const void* lq, const void* lk, int32_t* idx, float* sel,
                          hipStream_t st) {
  const int64_t ntq = (s.nQ + 63) / 64;
  const int64_t BHr = (int64_t)s.B * s.Hr;
  hipLaunchKernelGGL((fused_select_kernel<T, KM>), dim3((unsigned)(BHr * ntq)), dim3(256), 0, st, (const T*)lq,
                     (const T*)lk, idx, sel, s.nQ, s.nKV, s.D, s.score_scale, s.topk, ntq);
  note_launch("fused_select_kernel", st);
  return take_launch_error();
}

template <typename T>
hipError_t launch_scores_t(const Shape& s, const void* lq, const void* lk, float* scores, hipStream_t st) {
  const int64_t ntq = (s.nQ + 63) / 64, ntj = (s.nKV + 63) / 64;
  const int64_t nwork = (int64_t)s.B * s.Hr * ntq * ntj;
  hipLaunchKernelGGL(chunk_scores_kernel<T>, dim3((unsigned)round8(nwork)), dim3(256), 0, st,
                     (const T*)lq, (const T*)lk, scores, s.nQ, s.nKV, s.D, s.score_scale, s.causal, ntq,
                     ntj, nwork);
  note_launch("chunk_scores_kernel", st);
  return take_launch_error();
}

template <int KM>
hipError_t launch_topk_k(const Shape& s, const float* scores, int32_t* idx, float* sel, hipStream_t st) {
  const int64_t rows = (int64_t)s.B * s.Hr * s.nQ;
  hipLaunchKernelGGL(topk_kernel<KM>, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, scores, idx, sel,
                     rows, s.nQ, s.nKV, s.topk, s.causal);
  note_launch("topk_kernel", st);
  return take_launch_error();
}

template <typename T, int KM>
hipError_t launch_decode_k(const Shape& s, const void* lq, const void* lk, int32_t* idx, float* sel, void* ws,
                           hipStream_t st) {
  const ScanPlan plan = scan_plan(s.nKV);
  const int64_t rows = (int64_t)s.B * s.Hr;
  float* cs = reinterpret_cast<float*>(ws);
  int* cj = reinterpret_cast<int*>(reinterpret_cast<char*>(ws) +
                                   align256(sizeof(float) * rows * plan.slices * s.topk));
  const size_t smem = (size_t)s.D * sizeof(T);
  hipLaunchKernelGGL((decode_scan_kernel<T, KM>), dim3((unsigned)(rows * plan.slices)), dim3(kScanThreads), smem,
                     st, (const T*)lq, (const T*)lk, cs, cj, s.nKV, s.D, s.score_scale, s.topk, plan.per,
                     plan.slices);
  note_launch("decode_scan_kernel", st);
  const hipError_t e = take_launch_error();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_merge_kernel<KM>, dim3((unsigned)rows), dim3(kMergeThreads), 0, st, cs, cj, idx, sel, s.topk,
                     plan.slices);
  note_launch("decode_merge_kernel", st);
  return take_launch_error();
}

}  // namespace

hipError_t launch_chunk_scores(const Shape& s, const void* lmk_q, const void* lmk_k, float* scores,
                               hipStream_t stream) {
  return s.bf16 ? launch_scores_t<__bf16>(s, lmk_q, lmk_k, scores, stream)
                : launch_scores_t<float>(s, lmk_q, lmk_k, scores, stream);
}

hipError_t launch_topk(const Shape& s, const float* scores, int32_t* idx, float* sel, hipStream_t stream) {
  if (s.topk <= 8) return launch_topk_k<8>(s, scores, idx, sel, stream);
  if (s.topk <= 16) return launch_topk_k<16>(s, scores, idx, sel, stream);
  return launch_topk_k<32>(s, scores, idx, sel, stream);
}

size_t decode_workspace(const Shape& s) {
  const ScanPlan plan = scan_plan(s.nKV);
  const size_t n = (size_t)s.B * s.Hr * plan.slices * s.topk;
  return align256(n * sizeof(float)) + align256(n * sizeof(int));
}

hipError_t launch_decode_select(const Shape& s, const void* lmk_q, const void* lmk_k, int32_t* idx, float* sel,
                                void* ws, hipStream_t stream) {
  if (s.bf16) {
    if (s.topk <= 8) return launch_decode_k<__bf16, 8>(s, lmk_q, lmk_k, idx, sel, ws, stream);
    if (s.topk <= 16) return launch_decode_k<__bf16, 16>(s, lmk_q, lmk_k, idx, sel, ws, stream);
    return launch_decode_k<__bf16, 32>(s, lmk_q, lmk_k, idx, sel, ws, stream);
  }
  if (s.topk <= 8) return launch_decode_k<float, 8>(s, lmk_q, lmk_k, idx, sel, ws, stream);
  if (s.topk <= 16) return launch_decode_k<float, 16>(s, lmk_q, lmk_k, idx, sel, ws, stream);
  return launch_decode_k<float, 32>(s, lmk_q, lmk_k, idx, sel, ws, stream);
}

size_t fused_workspace(const Shape&) { return 0; }

hipError_t launch_fused_select(const Shape& s, const void* lmk_q, const void* lmk_k, int32_t* idx, float* sel,
                               void* ws, hipStream_t stream) {
  (void)ws;
  if (s.bf16) {
    if (s.topk <= 8) return launch_fused_k<__bf16, 8>(s, lmk_q, lmk_k, idx, sel, stream);
    if (s.topk <= 16) return launch_fused_k<__bf16, 16>(s, lmk_q, lmk_k, idx, sel, stream);
    return launch_fused_k<__bf16, 32>(s, lmk_q, lmk_k, idx, sel, stream);
  }
  if (s.topk <= 8) return launch_fused_k<float, 8>(s, lmk_q, lmk_k, idx, sel, stream);
  if (s.topk <= 16) return launch_fused_k<float, 16>(s, lmk_q, lmk_k, idx, sel, stream);
  return launch_fused_k<float, 32>(s, lmk_q, lmk_k, idx, sel, stream);
}

}  // namespace gca
