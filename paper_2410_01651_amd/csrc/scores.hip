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
// decode scan: one landmark query against every past landmark key.  The keys
//   are streamed once, coalesced, by ~256 workgroups whose waves each own a
//   contiguous range; 8 lanes share one key row and reduce the dot product
//   with three cross-lane steps.  Each wave leaves its range's best k in the
//   workspace; the decode attention kernel merges them (xattn_decode.hip).
#include "gca_device.hpp"
#include "gca_launch.hpp"

#include <type_traits>

namespace gca {
namespace {

// ------------------------------------------------------------ scores ----

// One 64x64 block of scores: landmark query rows a[0..63] against landmark key
// rows b[0..63] (rows at and past a_n / b_n repeat the last existing row; their
// scores are discarded by the caller), contracted over D in 64-column chunks.
// The workgroup copies each chunk of both row blocks into LDS with coalesced
// direct-to-LDS loads (128 contiguous bytes per row and copy), two stages deep,
// the next chunk in flight during the current chunk's products; wave w computes
// the 32x32 block of query rows 32 (w >> 1) and key rows 32 (w & 1).
template <typename T>
__device__ __forceinline__ f32x16 score_block(const T* a, int a_n, const T* b, int b_n, int D, T* stage) {
  constexpr int TILE = kS * kD;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
  const TileCopy<T, 4> ca(wave, lane, D, a_n), cb(wave, lane, D, b_n);
  constexpr int kLoads = 2 * TileCopy<T, 4>::kN;  // one wave's copies of one chunk
  const int nch = D / kD;
  auto issue = [&](int c) __device__ {
    T* st = stage + (c & 1) * 2 * TILE;
    ca.issue(a + c * kD, st);
    cb.issue(b + c * kD, st + TILE);
  };
  f32x16 acc = zero16();
  issue(0);
  for (int c = 0; c < nch; ++c) {
    if (c + 1 < nch) {
      issue(c + 1);
      wait_vmem<kLoads>();
    } else {
      wait_vmem<0>();
    }
    block_barrier();  // every wave's copies of chunk c are in
    const T* sa = stage + (c & 1) * 2 * TILE;
    const T* sb = sa + TILE;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      mma32(acc, lds_frag(sa, 32 * (wave >> 1) + (lane & 31), 16 * kb + 8 * hh),
            lds_frag(sb, 32 * (wave & 1) + (lane & 31), 16 * kb + 8 * hh));
    block_barrier();  // the stage is free for the copy issued in the next step
  }
  return acc;
}

template <typename T>
__global__ __launch_bounds__(256) void chunk_scores_kernel(const T* __restrict__ lq, const T* __restrict__ lk,
                                                           float* __restrict__ scores, int64_t nQ, int64_t nC,
                                                           int D, float scale, int causal, int64_t ntq,
                                                           int64_t ntj, int64_t nwork) {
  __shared__ __attribute__((aligned(16))) T stage[4 * kS * kD];
  const int64_t wid = xcd_swizzle(blockIdx.x, gridDim.x);
  if (wid >= nwork) return;
  const int64_t tj = wid % ntj;
  const int64_t rest = wid / ntj;
  const int64_t tq = rest % ntq;
  const int64_t bhr = rest / ntq;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
  const int64_t ta0 = tq * 64, tb0 = tj * 64;
  const int64_t t0 = ta0 + 32 * (wave >> 1);
  const int64_t j = tb0 + 32 * (wave & 1) + (lane & 31);
  float* out = scores + bhr * nQ * nC;

  f32x16 acc = zero16();
  // workgroup-uniform: the block holds some j < t (causal) and exists
  const bool live = ta0 < nQ && tb0 < nC && (!causal || tb0 < ta0 + 63);
  if (live)
    acc = score_block<T>(lq + (bhr * nQ + ta0) * D, (int)min<int64_t>(64, nQ - ta0), lk + (bhr * nC + tb0) * D,
                         (int)min<int64_t>(64, nC - tb0), D, stage);
  if (j < nC) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t t = t0 + 8 * (i >> 2) + 4 * hh + (i & 3);
      if (t < nQ) out[t * nC + j] = (live && (!causal || j < t)) ? acc[i] * scale : -INFINITY;
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

// GUMBEL: candidates are ranked by score + Gumbel noise; sel reports the raw
// score of each chosen chunk (read back from the matrix).
template <int KM, bool GUMBEL>
__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ scores, int32_t* __restrict__ idx,
                                                   float* __restrict__ sel, int64_t rows, int64_t nQ,
                                                   int64_t nC, int K, int causal, uint64_t seed) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t t = row % nQ;
  const int64_t lim = causal ? (t < nC ? t : nC) : nC;
  const float* sr = scores + row * nC;
  TopList<KM> L;
  L.init();
  // kTB scores per lane are loaded before they are inserted (in the same column
  // order), so a row of up to 64 kTB columns costs one memory latency (fewer
  // for the longer lists, whose unrolled inserts are larger)
  constexpr int kTB = KM <= 8 ? 16 : KM <= 16 ? 8 : 1;
  for (int64_t j0 = 0; j0 < lim; j0 += 64 * kTB) {
    float vb[kTB];
#pragma unroll
    for (int m = 0; m < kTB; ++m) {
      const int64_t j = j0 + 64 * m + lane;
      vb[m] = j < lim ? sr[j] : -INFINITY;
    }
#pragma unroll
    for (int m = 0; m < kTB; ++m) {
      const int64_t j = j0 + 64 * m + lane;
      float v = vb[m];
      if constexpr (GUMBEL) {
        if (j < lim) v += gumbel_noise(seed, (uint32_t)(row / nQ), (uint32_t)t, (uint32_t)j);
      }
      if (__builtin_isfinite(v)) L.insert(v, (int)j);  // columns past the row read -inf
    }
  }
  float ms;
  int mj, cnt;
  wave_merge(L, K, ms, mj, cnt);
  if constexpr (GUMBEL) ms = lane < cnt ? sr[mj] : -INFINITY;
  write_sorted<KM>(idx + row * K, sel + row * K, K, ms, mj, cnt);
}

// ------------------------------------------------------- decode scan ----

constexpr int kScanThreads = 256;
constexpr int kScanWaves = kScanThreads / 64;
static_assert(kScanWaves == kScanListWaves, "the merge's list mapping assumes four scan waves");
constexpr int kScanBatch = 8;  // column blocks per lane in one batch of loads

// Buffer descriptor over `bytes` bytes from `base` (wave-uniform): reads at
// offsets past the end return zero and touch no memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t range_rsrc(const char* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), 0, (int)bytes, 0x00020000);
}
constexpr int kLoadNonTemporal = 2;  // cache policy: streamed once

// Partial dot product of one lane's 8 elements of a key column block with the
// query's (both 16 bytes of bf16, or 32 bytes of fp32 as two records).
__device__ __forceinline__ float dot_block(const u32x4* v, const bf16x8 b, float acc) {
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
  const bf16x8 a = __builtin_bit_cast(bf16x8, v[0]);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 0, 1), __builtin_shufflevector(b, b, 0, 1),
                                        acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 2, 3), __builtin_shufflevector(b, b, 2, 3),
                                        acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 4, 5), __builtin_shufflevector(b, b, 4, 5),
                                        acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 6, 7), __builtin_shufflevector(b, b, 6, 7),
                                        acc, false);
  return acc;
}
__device__ __forceinline__ float dot_block(const u32x4* v, const f32x8 b, float acc) {
  const f32x4 a0 = __builtin_bit_cast(f32x4, v[0]), a1 = __builtin_bit_cast(f32x4, v[1]);
#pragma unroll
  for (int m = 0; m < 4; ++m) acc = fmaf(a0[m], b.lo[m], acc);
#pragma unroll
  for (int m = 0; m < 4; ++m) acc = fmaf(a1[m], b.hi[m], acc);
  return acc;
}

// Every workgroup scans one contiguous range of 4 pw landmark keys of its row:
// its four waves take the range's groups of 8 keys in turn (wave w: groups w,
// w + 4, ...), so the workgroup reads one stream (one stream per wave, 1,024 in
// all, measured 6-7 % slower), and each wave leaves the best k of its groups
// (sorted best first, padded with chunk -1) as list number (workgroup * 4 +
// wave) of the row.  8 lanes share a key: lane
// 8m + s reads bytes 16 s .. 16 s + 15 (bf16) of every 128-byte column block of
// key m of the current group of 8 keys, so one load instruction covers 8 keys x
// 128 contiguous bytes.  Loads are streamed (non-temporal) through a buffer
// descriptor per key group, whose range check zeroes the lanes past the end of
// the wave's range with no memory access, and run one batch of 8 column blocks
// ahead of the arithmetic.
// GUMBEL: the lists rank (and hold) score + Gumbel noise; the decode attention
// recomputes the chosen chunks' raw scores.  Q8 (D = 512, eight column blocks
// per key): every lane keeps its eight query fragments in registers, so there
// is no staging of the query through LDS and no barrier before the first loads,
// and a batch of loads is exactly one key group.
template <typename T, int KM, bool KEEP_ALL, bool GUMBEL, bool Q8>
__global__ __launch_bounds__(kScanThreads) void decode_scan_kernel(const T* __restrict__ lq,
                                                                   const T* __restrict__ lk, float* __restrict__ cs,
                                                                   int* __restrict__ cj, int64_t nC, int D,
                                                                   float scale, int K, int64_t pw, int64_t lists,
                                                                   int64_t wgs, uint64_t seed) {
  constexpr int LPS = (int)sizeof(T) / 2;  // 16-byte records per lane per column block
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  T* sq = reinterpret_cast<T*>(smem);

  const int64_t row = blockIdx.x / wgs, g = blockIdx.x % wgs;
  const int tid = threadIdx.x, lane = tid & 63, sub = lane & 7, kl = lane >> 3;
  const T* q = lq + row * D;  // the one landmark query of this row
  Frag<T> qreg[Q8 ? kScanBatch : 1];
  if constexpr (Q8) {
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) qreg[k] = load_frag(q + 64 * k + sub * 8);
  } else {
    for (int x = tid * (16 / (int)sizeof(T)); x < D; x += kScanThreads * (16 / (int)sizeof(T)))
      *reinterpret_cast<u32x4*>(sq + x) = *reinterpret_cast<const u32x4*>(q + x);
    __syncthreads();
  }

  const int wv = tid >> 6;
  const int64_t list = uniform64(g * kScanWaves + wv);
  if (list >= lists) return;
  // the workgroup's contiguous range of keys; this wave takes its key groups
  // wv, wv + 4, wv + 8, ... (group = 8 consecutive keys)
  const int64_t lo = g * kScanWaves * pw;
  const int64_t n = kScanWaves * pw < nC - lo ? kScanWaves * pw : nC - lo;  // keys in the range (>= 1)
  const int NB = D / 64;                          // column blocks per key
  const int64_t KB = (int64_t)D * sizeof(T);      // bytes per key
  const int64_t ngroups_wg = (n + 7) / 8;
  const int64_t ngroups = ngroups_wg > wv ? (ngroups_wg - wv + kScanWaves - 1) / kScanWaves : 0;
  auto key_of = [&](int64_t gi, int kk) { return 8 * (wv + kScanWaves * gi) + kk; };  // key of the range
  const int64_t nsteps = ngroups * NB;
  const int64_t nbatch = (nsteps + kScanBatch - 1) / kScanBatch;
  const char* const wbase = reinterpret_cast<const char*>(lk + (row * nC + lo) * D);
  const uint32_t lane_off = (uint32_t)(kl * KB) + (uint32_t)(sub * 16 * LPS);

  // issue cursor: key group ig, column block icb, and the group's descriptor
  int64_t ig = 0;
  int icb = 0;
  auto rsrc_of = [&](int64_t gi) {  // this wave's gi-th group
    const int64_t gg = wv + kScanWaves * gi;
    const int64_t left = (n - 8 * gg) * KB;
    const uint32_t bytes = left <= 0 ? 0u : (uint32_t)(left < 8 * KB ? left : 8 * KB);
    return range_rsrc(wbase + (left <= 0 ? 0 : gg * 8 * KB), bytes);
  };
  __amdgpu_buffer_rsrc_t rs = rsrc_of(0);
  auto issue = [&](u32x4* v) {
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
#pragma unroll
      for (int e = 0; e < LPS; ++e)
        v[k * LPS + e] = __builtin_amdgcn_raw_buffer_load_b128(rs, lane_off + 16 * e,
                                                               icb * 64 * (int)sizeof(T), kLoadNonTemporal);
      if (++icb == NB) {
        icb = 0;
        ++ig;
        rs = rsrc_of(ig);
      }
    }
  };

  // compute cursor
  int64_t cg = 0;
  int ccb = 0;
  float acc = 0.f;
  TopList<KM> L;
  L.init();
  // KEEP_ALL (a lane sees at most KM keys): lane (kl, sub) keeps the raw score
  // of key kl of the wave's group 8 m + sub in sc[m], ranked only at the end
  float sc[KEEP_ALL ? KM : 1];
  float mine = -INFINITY;
  if constexpr (KEEP_ALL) {
#pragma unroll
    for (int m = 0; m < KM; ++m) sc[m] = -INFINITY;
  }
  // the dot products of key group cg are complete in acc
  auto finish_group = [&]() {
    // sum over the key's 8 lanes (quad swaps, then the other quad)
    acc += dpp<kDppXor1>(acc);
    acc += dpp<kDppXor2>(acc);
    acc += dpp<kDppHalfMirror>(acc);
    if constexpr (KEEP_ALL) {
      if (sub == (int)(cg & 7)) mine = acc;
      if ((cg & 7) == 7 || cg + 1 == ngroups) {
#pragma unroll
        for (int m = 0; m < KM; ++m)
          if (m == (int)(cg >> 3)) sc[m] = mine;
        mine = -INFINITY;
      }
    } else {
      const int64_t key = key_of(cg, kl);
      // one of the key's 8 lanes inserts it, rotating with the group
      if (key < n && sub == (int)(cg & 7)) {
        float sv = acc * scale;
        if constexpr (GUMBEL) sv += gumbel_noise(seed, (uint32_t)row, 0u, (uint32_t)(lo + key));
        if (__builtin_isfinite(sv)) L.insert(sv, (int)(lo + key));
      }
    }
    acc = 0.f;
    ++cg;
  };
  auto consume = [&](const u32x4* v, int64_t step0) {
    if constexpr (Q8) {
      if (step0 < nsteps) {  // one whole group
#pragma unroll
        for (int k = 0; k < kScanBatch; ++k) acc = dot_block(v + k * LPS, qreg[k], acc);
        finish_group();
      }
    } else {
#pragma unroll
      for (int k = 0; k < kScanBatch; ++k) {
        if (step0 + k < nsteps) {
          acc = dot_block(v + k * LPS, load_frag(sq + ccb * 64 + sub * 8), acc);
          if (++ccb == NB) {
            ccb = 0;
            finish_group();
          }
        }
      }
    }
  };

  // two register batches alternate: batch b + 1 is in flight while batch b is
  // consumed; the loop body issues unconditionally so the waits stay exact
  u32x4 va[kScanBatch * LPS], vb[kScanBatch * LPS];
  issue(va);
  int64_t bt = 0;
  for (; bt + 2 < nbatch; bt += 2) {
    issue(vb);
    consume(va, bt * kScanBatch);
    issue(va);
    consume(vb, (bt + 1) * kScanBatch);
  }
  if (bt + 1 < nbatch) {
    issue(vb);
    consume(va, bt * kScanBatch);
    consume(vb, (bt + 1) * kScanBatch);
  } else {
    consume(va, bt * kScanBatch);
  }

  if constexpr (KEEP_ALL) {
#pragma unroll
    for (int m = 0; m < KM; ++m) {
      const int64_t key = key_of(8 * m + sub, kl);
      float sv = sc[m] * scale;
      if constexpr (GUMBEL) {
        if (key < n) sv += gumbel_noise(seed, (uint32_t)row, 0u, (uint32_t)(lo + key));
      }
      if (key < n && __builtin_isfinite(sv)) L.insert(sv, (int)(lo + key));
    }
  }
  float ms;
  int mj, cnt;
  wave_merge(L, K, ms, mj, cnt);
  if (lane < K) {
    const int64_t o = (row * lists + list) * K + lane;
    cs[o] = lane < cnt ? ms : -INFINITY;
    cj[o] = lane < cnt ? mj : -1;
  }
}

// ------------------------------------------------ fused causal select ----

// Scores and top-k in one pass for a block of 64 landmark rows: the workgroup
// walks the key tiles j < t in order, computes each 64x64 score tile on the
// matrix cores into LDS, and 4 threads per row fold the tile into their
// running best-KM lists.  No score matrix is written.  Row blocks are issued
// longest first (block tq has tq+1 tiles) so the triangular work balances.
// GUMBEL: the lists rank score + Gumbel noise (each thread then takes 16
// consecutive columns, four generator calls per tile) and the chosen chunks'
// raw scores are recomputed from the landmark rows for sel.
template <typename T, int KM, bool GUMBEL>
__global__ __launch_bounds__(256) void fused_select_kernel(const T* __restrict__ lq, const T* __restrict__ lk,
                                                           int32_t* __restrict__ idx, float* __restrict__ sel,
                                                           int64_t nQ, int64_t nC, int D, float scale, int K,
                                                           int64_t ntq, uint64_t seed) {
  __shared__ __attribute__((aligned(16))) T stage[4 * kS * kD];
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
    const f32x16 acc = score_block<T>(lq + (bhr * nQ + t0) * D, (int)min<int64_t>(64, nQ - t0),
                                      lk + (bhr * nC + j0) * D, (int)min<int64_t>(64, nC - j0), D, stage);
    const int jl = 32 * (wave & 1) + (lane & 31);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int tl = 32 * (wave >> 1) + 8 * (i >> 2) + 4 * hh + (i & 3);
      const int64_t t = t0 + tl, j = j0 + jl;
      sT[tl][jl] = (any && t < nQ && j < nC && j < t) ? acc[i] * scale : -INFINITY;
    }
    __syncthreads();
    if constexpr (GUMBEL) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int c0 = 16 * u + 4 * q4;
        const f32x4 g = gumbel_noise4(seed, (uint32_t)bhr, (uint32_t)(t0 + r), (uint32_t)((j0 + c0) >> 2));
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const float v = sT[r][c0 + m] + g[m];
          if (__builtin_isfinite(v)) L.insert(v, (int)(j0 + c0 + m));
        }
      }
    } else {
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        const int c = u + 4 * m;
        const float v = sT[r][c];
        if (__builtin_isfinite(v)) L.insert(v, (int)(j0 + c));
      }
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
        if constexpr (GUMBEL)
          so[rank] = scale * dot_rows(lq + (bhr * nQ + t) * D, lk + (bhr * nC + je) * D, D);
        else
          so[rank] = sRs[r][e];
      } else {
        io[e] = -1;
        so[e] = -INFINITY;
      }
    }
  }
}

template <typename T, int KM, bool GUMBEL>
hipError_t launch_fused_k(const Shape& s, const void* lq, const void* lk, int32_t* idx, float* sel,
                          hipStream_t st) {
  const int64_t ntq = (s.nQ + 63) / 64;
  const int64_t BHr = (int64_t)s.B * s.Hr;
  launch_kernel("fused_select_kernel", fused_select_kernel<T, KM, GUMBEL>, dim3((unsigned)(BHr * ntq)), dim3(256),
                0, st, (const T*)lq, (const T*)lk, idx, sel, s.nQ, s.nKV, s.D, s.score_scale, s.topk, ntq,
                s.gumbel_seed);
  return take_launch_error();
}

template <typename T>
hipError_t launch_scores_t(const Shape& s, const void* lq, const void* lk, float* scores, hipStream_t st) {
  const int64_t ntq = (s.nQ + 63) / 64, ntj = (s.nKV + 63) / 64;
  const int64_t nwork = (int64_t)s.B * s.Hr * ntq * ntj;
  launch_kernel("chunk_scores_kernel", chunk_scores_kernel<T>, dim3((unsigned)round8(nwork)), dim3(256), 0, st,
                (const T*)lq, (const T*)lk, scores, s.nQ, s.nKV, s.D, s.score_scale, s.causal, ntq, ntj, nwork);
  return take_launch_error();
}

template <int KM, bool GUMBEL>
hipError_t launch_topk_k(const Shape& s, const float* scores, int32_t* idx, float* sel, hipStream_t st) {
  const int64_t rows = (int64_t)s.B * s.Hr * s.nQ;
  launch_kernel("topk_kernel", topk_kernel<KM, GUMBEL>, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, scores,
                idx, sel, rows, s.nQ, s.nKV, s.topk, s.causal, s.gumbel_seed);
  return take_launch_error();
}

template <typename T, int KM, bool KEEP_ALL, bool GUMBEL, bool Q8>
hipError_t launch_scan_q(const Shape& s, const void* lq, const void* lk, void* ws, hipStream_t st) {
  const DecodePlan plan = decode_plan(s);
  const int64_t rows = (int64_t)s.B * s.Hr;
  float* cs = decode_list_scores(s, ws);
  int* cj = decode_list_chunks(s, ws);
  const size_t smem = Q8 ? 0 : (size_t)s.D * sizeof(T);
  launch_kernel("decode_scan_kernel", decode_scan_kernel<T, KM, KEEP_ALL, GUMBEL, Q8>,
                dim3((unsigned)(rows * plan.wgs)), dim3(kScanThreads), smem, st, (const T*)lq, (const T*)lk, cs, cj, s.nKV, s.D, s.score_scale, s.topk,
                plan.pw, plan.lists, plan.wgs, s.gumbel_seed);
  return take_launch_error();
}

template <typename T, int KM, bool KEEP_ALL, bool GUMBEL>
hipError_t launch_scan_k(const Shape& s, const void* lq, const void* lk, void* ws, hipStream_t st) {
  if (s.D == 64 * kScanBatch) return launch_scan_q<T, KM, KEEP_ALL, GUMBEL, true>(s, lq, lk, ws, st);
  return launch_scan_q<T, KM, KEEP_ALL, GUMBEL, false>(s, lq, lk, ws, st);
}

}  // namespace

hipError_t launch_chunk_scores(const Shape& s, const void* lmk_q, const void* lmk_k, float* scores,
                               hipStream_t stream) {
  return s.bf16 ? launch_scores_t<__bf16>(s, lmk_q, lmk_k, scores, stream)
                : launch_scores_t<float>(s, lmk_q, lmk_k, scores, stream);
}

hipError_t launch_topk(const Shape& s, const float* scores, int32_t* idx, float* sel, hipStream_t stream) {
  auto run = [&](auto gumbel) {
    constexpr bool G = decltype(gumbel)::value;
    if (s.topk <= 8) return launch_topk_k<8, G>(s, scores, idx, sel, stream);
    if (s.topk <= 16) return launch_topk_k<16, G>(s, scores, idx, sel, stream);
    return launch_topk_k<32, G>(s, scores, idx, sel, stream);
  };
  return s.gumbel ? run(std::true_type{}) : run(std::false_type{});
}

hipError_t launch_decode_scan(const Shape& s, const void* lmk_q, const void* lmk_k, void* ws, hipStream_t stream) {
  // A lane sees at most ceil(pw / 64) keys of its wave's range (one key of every
  // eighth group of 8).  Up to k of them it keeps every raw score and ranks them
  // at the end; beyond, it keeps a running best-k list.
  const int64_t per_lane = (decode_plan(s).pw + 63) / 64;
  auto run = [&](auto tag, auto gumbel) {
    using T = decltype(tag);
    constexpr bool G = decltype(gumbel)::value;
    if (per_lane <= s.topk) {
      if (per_lane <= 1) return launch_scan_k<T, 1, true, G>(s, lmk_q, lmk_k, ws, stream);
      if (per_lane <= 2) return launch_scan_k<T, 2, true, G>(s, lmk_q, lmk_k, ws, stream);
      if (per_lane <= 4) return launch_scan_k<T, 4, true, G>(s, lmk_q, lmk_k, ws, stream);
      if (per_lane <= 8) return launch_scan_k<T, 8, true, G>(s, lmk_q, lmk_k, ws, stream);
      if (per_lane <= 16) return launch_scan_k<T, 16, true, G>(s, lmk_q, lmk_k, ws, stream);
      return launch_scan_k<T, 32, true, G>(s, lmk_q, lmk_k, ws, stream);
    }
    if (s.topk <= 8) return launch_scan_k<T, 8, false, G>(s, lmk_q, lmk_k, ws, stream);
    if (s.topk <= 16) return launch_scan_k<T, 16, false, G>(s, lmk_q, lmk_k, ws, stream);
    return launch_scan_k<T, 32, false, G>(s, lmk_q, lmk_k, ws, stream);
  };
  if (s.bf16) return s.gumbel ? run(__bf16{}, std::true_type{}) : run(__bf16{}, std::false_type{});
  return s.gumbel ? run(float{}, std::true_type{}) : run(float{}, std::false_type{});
}

hipError_t launch_fused_rowblocks(const Shape& s, const void* lmk_q, const void* lmk_k, int32_t* idx, float* sel,
                                  hipStream_t stream) {
  auto run = [&](auto tag, auto gumbel) {
    using T = decltype(tag);
    constexpr bool G = decltype(gumbel)::value;
    if (s.topk <= 8) return launch_fused_k<T, 8, G>(s, lmk_q, lmk_k, idx, sel, stream);
    if (s.topk <= 16) return launch_fused_k<T, 16, G>(s, lmk_q, lmk_k, idx, sel, stream);
    return launch_fused_k<T, 32, G>(s, lmk_q, lmk_k, idx, sel, stream);
  };
  if (s.bf16) return s.gumbel ? run(__bf16{}, std::true_type{}) : run(__bf16{}, std::false_type{});
  return s.gumbel ? run(float{}, std::true_type{}) : run(float{}, std::false_type{});
}

}  // namespace gca
