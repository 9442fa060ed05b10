// Backward of grouped cross attention (Algorithm 2 of the method's appendix)
// and of the retrieval scores (Eq. 2) and landmark vectors (Eq. 1).
//
// With P_s = softmax of one (query chunk, retrieved chunk j) tile, recomputed
// from the saved log-sum-exp, dP_s = dO V_j^T, D_s = rowsum(P_s o dP_s) and
// dS_s = w_s P_s o (dP_s - D_s):
//   dQ_c  += scale * dS_s K_j           (query-stationary kernel)
//   dV_j  += (w_s P_s)^T dO_c           (key-stationary kernel)
//   dK_j  += scale * dS_s^T Q_c         (key-stationary kernel)
//   dw[t,s] = sum over the group's heads and the chunk's rows of D_s
// D_s equals rowsum(dO o O'_s) of Algorithm 2, computed here on chip from the
// same tile, so the per-chunk outputs O'_s are never stored.
//
// No floating-point atomics: every output element is produced by exactly one
// workgroup.  The key-stationary pass needs, for each chunk j, the list of
// (row t, slot s) that retrieved it; an integer counting sort builds that list
// (CSR) and a rank pass orders each list by (t, s), so the summation order, and
// hence the result, is the same on every run.
#include "gca_device.hpp"
#include "gca_launch.hpp"

#include <algorithm>
#include <type_traits>

namespace gca {
namespace {

constexpr int kThreads = 256;  // two pairs of waves

template <typename T> struct LdsLd;
template <> struct LdsLd<__bf16> { static constexpr int v = 72; };
template <> struct LdsLd<float> { static constexpr int v = 68; };

struct Ws {
  float* w;        // [B*Hr, nQ, K] fusion weights
  float* Dbuf;     // [B*H, Lq, K]  D_s per query token
  float* dwp;      // [B*H, nQ, K]  per-head dw partials
  int* counts;     // [B*Hr, nKV]
  int* cursor;     // [B*Hr, nKV]
  int* offs;       // [B*Hr, nKV+1]
  int* unsorted;   // [B*Hr, nQ*K]
  int* sorted;     // [B*Hr, nQ*K]
};

Ws carve(const Shape& s, void* base) {
  const int64_t BHr = (int64_t)s.B * s.Hr, BH = (int64_t)s.B * s.H;
  char* p = reinterpret_cast<char*>(base);
  Ws w;
  auto take = [&](size_t bytes) { char* r = p; p += align256(bytes); return r; };
  w.w = (float*)take(sizeof(float) * BHr * s.nQ * s.topk);
  w.Dbuf = (float*)take(sizeof(float) * BH * s.nQ * kS * s.topk);
  w.dwp = (float*)take(sizeof(float) * BH * s.nQ * s.topk);
  w.counts = (int*)take(sizeof(int) * BHr * s.nKV);
  w.cursor = (int*)take(sizeof(int) * BHr * s.nKV);
  w.offs = (int*)take(sizeof(int) * BHr * (s.nKV + 1));
  w.unsorted = (int*)take(sizeof(int) * BHr * s.nQ * s.topk);
  w.sorted = (int*)take(sizeof(int) * BHr * s.nQ * s.topk);
  return w;
}

size_t carve_size(const Shape& s) {
  const int64_t BHr = (int64_t)s.B * s.Hr, BH = (int64_t)s.B * s.H;
  size_t n = 0;
  n += align256(sizeof(float) * BHr * s.nQ * s.topk);
  n += align256(sizeof(float) * BH * s.nQ * kS * s.topk);
  n += align256(sizeof(float) * BH * s.nQ * s.topk);
  n += align256(sizeof(int) * BHr * s.nKV) * 2;
  n += align256(sizeof(int) * BHr * (s.nKV + 1));
  n += align256(sizeof(int) * BHr * s.nQ * s.topk) * 2;
  return n;
}

struct BwdParams {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* idx;
  const float* sel;
  const float* lse;
  const void* dout;
  void* dq;
  void* dk;
  void* dv;
  Ws ws;
  int B, H, Hr, K;
  int64_t nQ, nKV;
  int causal;
  float attn_scale;
};

// ------------------------------------------------------------ helpers ----

__global__ void fill_zero_kernel(int* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

// Fusion weights of every retrieval row (Eq. 2), as the forward computed them.
__global__ void weights_kernel(const int32_t* __restrict__ idx, const float* __restrict__ sel,
                               float* __restrict__ w, int64_t rows, int K, int64_t nKV) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= rows * K) return;
  const int64_t row = e / K;
  const int s = (int)(e % K);
  float wv;
  int jv;
  row_weight(idx + row * K, sel + row * K, K, nKV, s, wv, jv);
  w[e] = wv;
}

// ----------------------------------------------------- inverse index ----

// An entry (t, s) is listed under chunk idx[t, s] when row t feeds a query
// chunk that exists (causal: t + 1 < nQ; decode: t == 0).
__device__ __forceinline__ bool entry_live(int64_t t, int64_t nQ, int causal) {
  return t + causal < nQ;
}

__global__ void csr_count_kernel(const int32_t* __restrict__ idx, int* __restrict__ counts, int64_t BHr,
                                 int64_t nQ, int K, int64_t nKV, int causal) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= BHr * nQ * K) return;
  const int64_t bhr = e / (nQ * K);
  const int64_t t = (e / K) % nQ;
  const int j = idx[e];
  if (j >= 0 && j < nKV && entry_live(t, nQ, causal)) atomicAdd(&counts[bhr * nKV + j], 1);
}

// Exclusive scan of one (b, hr) count row: offs[0..nKV], cursor = offs[0..nKV).
__global__ __launch_bounds__(1024) void csr_scan_kernel(const int* __restrict__ counts, int* __restrict__ offs,
                                                        int* __restrict__ cursor, int64_t nKV) {
  __shared__ int sWave[16];
  __shared__ int sCarry;
  const int64_t bhr = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int* cnt = counts + bhr * nKV;
  int* off = offs + bhr * (nKV + 1);
  int* cur = cursor + bhr * nKV;
  if (tid == 0) sCarry = 0;
  __syncthreads();
  for (int64_t base = 0; base < nKV; base += 1024) {
    const int64_t i = base + tid;
    const int v = i < nKV ? cnt[i] : 0;
    int x = v;  // inclusive scan within the wave
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) sWave[wave] = x;
    __syncthreads();
    int before = sCarry;
    for (int w = 0; w < wave; ++w) before += sWave[w];
    const int excl = before + x - v;
    if (i < nKV) {
      off[i] = excl;
      cur[i] = excl;
    }
    __syncthreads();
    if (tid == 1023) sCarry = excl + v;
    __syncthreads();
  }
  if (tid == 0) off[nKV] = sCarry;
}

__global__ void csr_fill_kernel(const int32_t* __restrict__ idx, int* __restrict__ cursor,
                                int* __restrict__ unsorted, int64_t BHr, int64_t nQ, int K, int64_t nKV,
                                int causal) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= BHr * nQ * K) return;
  const int64_t bhr = e / (nQ * K);
  const int64_t local = e % (nQ * K);  // t * K + s
  const int64_t t = local / K;
  const int j = idx[e];
  if (j >= 0 && j < nKV && entry_live(t, nQ, causal)) {
    const int pos = atomicAdd(&cursor[bhr * nKV + j], 1);
    unsorted[bhr * nQ * K + pos] = (int)local;
  }
}

// Order each chunk's list ascending by (t, s): an entry's position is the number
// of smaller entries in its list (entries are distinct).  One wave per chunk.
__global__ __launch_bounds__(256) void csr_sort_kernel(const int* __restrict__ offs, const int* __restrict__ unsorted,
                                                       int* __restrict__ sorted, int64_t BHr, int64_t nQ, int K,
                                                       int64_t nKV) {
  const int64_t wv = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wv >= BHr * nKV) return;
  const int lane = threadIdx.x & 63;
  const int64_t bhr = wv / nKV, j = wv % nKV;
  const int* off = offs + bhr * (nKV + 1);
  const int lo = off[j], hi = off[j + 1];
  const int* src = unsorted + bhr * nQ * K;
  int* dst = sorted + bhr * nQ * K;
  for (int i = lo + lane; i < hi; i += 64) {
    const int e = src[i];
    int rank = 0;
    for (int u = lo; u < hi; ++u) rank += src[u] < e ? 1 : 0;
    dst[lo + rank] = e;
  }
}

// ------------------------------------------------- query-stationary dQ ----

// One workgroup of four waves per (batch, head, query chunk); the two wave pairs
// take alternate retrieved chunks from a four-slot LDS ring (K_j and V_j tiles),
// each wave owning 32 query tokens.  dQ partials of the pairs are summed at the end.
template <typename T>
__global__ __launch_bounds__(kThreads) void bwd_dq_kernel(BwdParams p, int64_t nwork) {
  constexpr int TILE = kS * kD;
  GCA_RING4(T, 2 * TILE)
  __shared__ float sL[32 * kS];  // [slot][query]: lse on entry, D_s on exit
  __shared__ float sW[32];
  __shared__ int sJ[32];
  __shared__ int sSlot[32];
  __shared__ int sN;

  const int64_t wid = xcd_swizzle(blockIdx.x, gridDim.x);
  if (wid >= nwork) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5;
  const int pair = wave >> 1, half = wave & 1;
  const int64_t c = wid % p.nQ;
  const int64_t bh = wid / p.nQ;
  const int h = (int)(bh % p.H);
  const int64_t b = bh / p.H;
  const int hr = p.Hr == 1 ? 0 : h;
  const int64_t t = p.causal ? c - 1 : 0;
  const int K = p.K;
  const int64_t row_base = (b * p.Hr + hr) * p.nQ;
  const int64_t tok0 = ((b * p.H + h) * p.nQ + c) * kS;

  if (wave == 0) {
    int jv = -1;
    float wv = 0.f;
    if (t >= 0 && lane < K) {
      const int j = p.idx[(row_base + t) * K + lane];
      if (j >= 0 && j < p.nKV) {
        jv = j;
        wv = p.ws.w[(row_base + t) * K + lane];
      }
    }
    const uint64_t mask = __ballot(jv >= 0);
    if (lane < 32) {
      sW[lane] = wv;
      sJ[lane] = jv;
    }
    if (jv >= 0) sSlot[__popcll(mask & ((1ull << lane) - 1))] = lane;
    if (lane == 0) sN = __popcll(mask);
  }
  if (t >= 0)
    for (int s = wave; s < K; s += 4) sL[s * kS + lane] = p.lse[(tok0 + lane) * K + s];
  __syncthreads();
  const int n = sN;
  // lane u < 32 holds valid item u's slot, chunk and weight (picked with a lane read)
  const int ls = sSlot[lane & 31] & 31;
  const int lj = sJ[ls];
  const float lw = sW[ls];

  T* dq = reinterpret_cast<T*>(p.dq) + tok0 * kD;
  if (n == 0) {
    for (int e = tid; e < kS * kD / 4; e += kThreads) store4(dq + 4 * e, 0.f, 0.f, 0.f, 0.f);
    if (t >= 0 && tid < K) p.ws.dwp[(bh * p.nQ + t) * K + tid] = 0.f;
    return;
  }

  const int qi = 32 * half + (lane & 31);
  const T* qrow = reinterpret_cast<const T*>(p.q) + (tok0 + qi) * kD;
  const T* dorow = reinterpret_cast<const T*>(p.dout) + (tok0 + qi) * kD;
  Frag<T> qf[4], df[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    qf[kb] = load_frag(qrow + 16 * kb + 8 * hh);
    df[kb] = load_frag(dorow + 16 * kb + 8 * hh);
  }
  wait_vmem<0>();

  const int64_t kv0 = (b * p.H + h) * p.nKV * TILE;
  const T* kbase = reinterpret_cast<const T*>(p.k) + kv0;
  const T* vbase = reinterpret_cast<const T*>(p.v) + kv0;
  f32x16 g0 = zero16(), g1 = zero16();  // dQ^T, d rows 0-31 / 32-63
  const float sc = p.attn_scale * kLog2e;
  const int cb = 16 * ((lane >> 4) & 1);

  const TileCopy<T, 4> cp(wave, lane);
  auto issue = [&](auto B, int u) __device__ {
    const int64_t j = __builtin_amdgcn_readlane(lj, u);
    T* dst = slot_buf(B);
    cp.issue(kbase + j * TILE, dst);
    cp.issue(vbase + j * TILE, dst + TILE);
  };
  auto run = [&](auto B, int u) __device__ {
    const int s = __builtin_amdgcn_readlane(ls, u);
    const T* sK = slot_buf(B);
    const T* sV = sK + TILE;
    const float lse2 = sL[s * kS + qi] * kLog2e;
    f32x16 s0 = zero16(), s1 = zero16(), p0 = zero16(), p1 = zero16();
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      mma32(s0, lds_frag(sK, lane & 31, 16 * kb + 8 * hh), qf[kb]);
      mma32(s1, lds_frag(sK, 32 + (lane & 31), 16 * kb + 8 * hh), qf[kb]);
      mma32(p0, lds_frag(sV, lane & 31, 16 * kb + 8 * hh), df[kb]);
      mma32(p1, lds_frag(sV, 32 + (lane & 31), 16 * kb + 8 * hh), df[kb]);
    }
    // P^T and D = rowsum(P o dP) for this lane's query
    float Dq = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      s0[i] = __builtin_amdgcn_exp2f(fmaf(s0[i], sc, -lse2));
      s1[i] = __builtin_amdgcn_exp2f(fmaf(s1[i], sc, -lse2));
      Dq += s0[i] * p0[i] + s1[i] * p1[i];
    }
    Dq = sum_xor32(Dq);
    if (hh == 0) sL[s * kS + qi] = Dq;  // this lane's pair alone reads the lse it replaces
    const float ws = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lw), u));
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      s0[i] = ws * s0[i] * (p0[i] - Dq);
      s1[i] = ws * s1[i] * (p1[i] - Dq);
    }
    Frag<T> f[4];
    frag_from_acc(f[0], s0, 0, 1.f);
    frag_from_acc(f[1], s0, 1, 1.f);
    frag_from_acc(f[2], s1, 0, 1.f);
    frag_from_acc(f[3], s1, 1, 1.f);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      mma32(g0, lds_frag_t(sK, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb), f[kb]);
      mma32(g1, lds_frag_t(sK, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb), f[kb]);
    }
  };
  pair_ring(n, pair, issue, run);

  // pair 1 hands its dQ^T partial to pair 0 through LDS, laid out
  // [half][register group][d half][lane] so that every access is lane-contiguous
  float* part = reinterpret_cast<float*>(ring0);
  auto part_at = [&](int g, int dt) { return part + ((half * 4 + g) * 2 + dt) * 256 + lane * 4; };
  __syncthreads();
  if (pair == 1) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      *reinterpret_cast<f32x4*>(part_at(g, 0)) = f32x4{g0[4 * g], g0[4 * g + 1], g0[4 * g + 2], g0[4 * g + 3]};
      *reinterpret_cast<f32x4*>(part_at(g, 1)) = f32x4{g1[4 * g], g1[4 * g + 1], g1[4 * g + 2], g1[4 * g + 3]};
    }
  }
  __syncthreads();
  if (pair == 0) {
    const float as = p.attn_scale;
    T* drow = dq + qi * kD;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(part_at(g, 0));
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(part_at(g, 1));
      store4(drow + 8 * g + 4 * hh, as * (g0[4 * g] + x0[0]), as * (g0[4 * g + 1] + x0[1]),
             as * (g0[4 * g + 2] + x0[2]), as * (g0[4 * g + 3] + x0[3]));
      store4(drow + 32 + 8 * g + 4 * hh, as * (g1[4 * g] + x1[0]), as * (g1[4 * g + 1] + x1[1]),
             as * (g1[4 * g + 2] + x1[2]), as * (g1[4 * g + 3] + x1[3]));
    }
  }
  // dw[t, s] = sum over the chunk's 64 queries of D_s (staged in sL): one wave per slot
  for (int s = wave; s < K; s += 4) {
    float acc = sJ[s] >= 0 ? sL[s * kS + lane] : 0.f;
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) acc += __shfl_xor(acc, o);
    acc = sum_xor32(acc);
    if (lane == 0) p.ws.dwp[(bh * p.nQ + t) * K + s] = acc;
  }
  float* Dout = p.ws.Dbuf + (tok0 + lane) * K;
  for (int s = wave; s < K; s += 4) Dout[s] = sJ[s] >= 0 ? sL[s * kS + lane] : 0.f;
}

// ---------------------------------------------- key-stationary dK, dV ----

// One workgroup of four waves per (batch, head, key chunk j); the two wave pairs
// take alternate retrievers (row t, slot s) of chunk j from a four-slot LDS ring
// (Q_c and dO_c tiles plus the lse and D columns of slot s), each wave owning 32
// of chunk j's keys.  dK/dV partials of the pairs are summed at the end.
template <typename T>
__global__ __launch_bounds__(kThreads, 2) void bwd_dkdv_kernel(BwdParams p, int64_t nwork) {
  constexpr int TILE = kS * kD;
  // ring slot: Q_c tile, dO_c tile, lse column, D column
  constexpr int ENTRY = 2 * TILE + 2 * kS * (int)(sizeof(float) / sizeof(T));
  __shared__ __attribute__((aligned(16))) T ring[4 * ENTRY];
  constexpr int NE = 256;  // retrievers staged in LDS per batch
  __shared__ int sE[NE];
  __shared__ float sWt[NE];

  const int64_t wid = xcd_swizzle(blockIdx.x, gridDim.x);
  if (wid >= nwork) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5;
  const int pair = wave >> 1, half = wave & 1;
  const int64_t j = wid % p.nKV;
  const int64_t bh = wid / p.nKV;
  const int h = (int)(bh % p.H);
  const int64_t b = bh / p.H;
  const int hr = p.Hr == 1 ? 0 : h;
  const int K = p.K;
  const int64_t bhr = b * p.Hr + hr;
  const int* off = p.ws.offs + bhr * (p.nKV + 1);
  const int lo = off[j], hi = off[j + 1];
  const int* list_g = p.ws.sorted + bhr * p.nQ * K + lo;
  const int n = hi - lo;

  const int64_t key0 = (bh * p.nKV + j) * kS;  // first key token of chunk j
  T* dk = reinterpret_cast<T*>(p.dk) + key0 * kD;
  T* dv = reinterpret_cast<T*>(p.dv) + key0 * kD;
  if (n == 0) {
    for (int e = tid; e < kS * kD / 4; e += kThreads) {
      store4(dk + 4 * e, 0.f, 0.f, 0.f, 0.f);
      store4(dv + 4 * e, 0.f, 0.f, 0.f, 0.f);
    }
    return;
  }

  // this wave's 32 keys of chunk j as B operands (K^T, V^T columns)
  const int kr = 32 * half + (lane & 31);
  const T* krow = reinterpret_cast<const T*>(p.k) + (key0 + kr) * kD;
  const T* vrow = reinterpret_cast<const T*>(p.v) + (key0 + kr) * kD;
  Frag<T> kf[4], vf[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    kf[kb] = load_frag(krow + 16 * kb + 8 * hh);
    vf[kb] = load_frag(vrow + 16 * kb + 8 * hh);
  }
  wait_vmem<0>();

  const T* qb = reinterpret_cast<const T*>(p.q) + bh * p.nQ * kS * kD;
  const T* ob = reinterpret_cast<const T*>(p.dout) + bh * p.nQ * kS * kD;
  const float* lseb = p.lse + bh * p.nQ * kS * K;
  const float* Db = p.ws.Dbuf + bh * p.nQ * kS * K;
  const float* wrow = p.ws.w + bhr * p.nQ * K;

  const TileCopy<T, 4> cp(wave, lane);
  const uint32_t col_off = (uint32_t)(lane * K * sizeof(float));
  auto issue = [&](int slot, int u) __device__ {
    const int cs = sE[u];  // (query chunk << 5) | slot
    const int64_t c = cs >> 5;
    const int s = cs & 31;
    T* dst = ring + slot * ENTRY;
    cp.issue(qb + c * TILE, dst);
    cp.issue(ob + c * TILE, dst + TILE);
    float* cols = reinterpret_cast<float*>(dst + 2 * TILE);
    if (wave == 0) dma_column_s(lseb + c * kS * K + s, col_off, cols);
    else if (wave == 1) dma_column_s(Db + c * kS * K + s, col_off, cols + kS);
  };

  f32x16 dv0 = zero16(), dv1 = zero16(), dk0 = zero16(), dk1 = zero16();
  const float sc = p.attn_scale * kLog2e;
  const int cb = 16 * ((lane >> 4) & 1);

  auto run = [&](int slot, int u) __device__ {
    const float wt = sWt[u];
    const T* sQ = ring + slot * ENTRY;
    const T* sO = sQ + TILE;
    const float* sL = reinterpret_cast<const float*>(sQ + 2 * TILE);
    const float* sD = sL + kS;
    // S = Q K^T for this wave's keys; queries 0-31 in s0, 32-63 in s1
    Frag<T> wp[4];
    {
      f32x16 s0 = zero16(), s1 = zero16();
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        mma32(s0, lds_frag(sQ, lane & 31, 16 * kb + 8 * hh), kf[kb]);
        mma32(s1, lds_frag(sQ, 32 + (lane & 31), 16 * kb + 8 * hh), kf[kb]);
      }
      // w P; accumulator row i holds query 32*qt + 8*(i/4) + 4*hh + i%4
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 l0 = *reinterpret_cast<const f32x4*>(sL + 8 * g + 4 * hh);
        const f32x4 l1 = *reinterpret_cast<const f32x4*>(sL + 32 + 8 * g + 4 * hh);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          s0[4 * g + r] = wt * __builtin_amdgcn_exp2f(fmaf(s0[4 * g + r], sc, -l0[r] * kLog2e));
          s1[4 * g + r] = wt * __builtin_amdgcn_exp2f(fmaf(s1[4 * g + r], sc, -l1[r] * kLog2e));
        }
      }
      frag_from_acc(wp[0], s0, 0, 1.f);
      frag_from_acc(wp[1], s0, 1, 1.f);
      frag_from_acc(wp[2], s1, 0, 1.f);
      frag_from_acc(wp[3], s1, 1, 1.f);
    }
    // dV^T += dO^T (w P)  (contraction over the 64 queries)
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      mma32(dv0, lds_frag_t(sO, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb), wp[kb]);
      mma32(dv1, lds_frag_t(sO, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb), wp[kb]);
    }
    // dP = dO V^T, then dS = w P o (dP - D) from the w P fragments
    Frag<T> ds[4];
    {
      f32x16 p0 = zero16(), p1 = zero16();
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        mma32(p0, lds_frag(sO, lane & 31, 16 * kb + 8 * hh), vf[kb]);
        mma32(p1, lds_frag(sO, 32 + (lane & 31), 16 * kb + 8 * hh), vf[kb]);
      }
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 d0 = *reinterpret_cast<const f32x4*>(sD + 8 * g + 4 * hh);
        const f32x4 d1 = *reinterpret_cast<const f32x4*>(sD + 32 + 8 * g + 4 * hh);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = 4 * g + r;  // register i of tile qt lives in wp[2*qt + i/8] entry i%8
          p0[i] = frag_elem(wp[i >> 3], i & 7) * (p0[i] - d0[r]);
          p1[i] = frag_elem(wp[2 + (i >> 3)], i & 7) * (p1[i] - d1[r]);
        }
      }
      frag_from_acc(ds[0], p0, 0, 1.f);
      frag_from_acc(ds[1], p0, 1, 1.f);
      frag_from_acc(ds[2], p1, 0, 1.f);
      frag_from_acc(ds[3], p1, 1, 1.f);
    }
    // dK^T += Q^T dS
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      mma32(dk0, lds_frag_t(sQ, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb), ds[kb]);
      mma32(dk1, lds_frag_t(sQ, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb), ds[kb]);
    }
  };

  // the retriever list is staged through LDS in batches, each streamed through
  // the ring and drained at its end
  for (int b0 = 0; b0 < n; b0 += NE) {
    const int nb = min(NE, n - b0);
    __syncthreads();
    for (int i = tid; i < nb; i += kThreads) {
      const int e = list_g[b0 + i];  // t * K + s
      sE[i] = ((e / K + p.causal) << 5) | (e % K);
      sWt[i] = wrow[e];
    }
    __syncthreads();
    pair_ring_dyn(nb, pair, issue, run);
  }

  // pair 1 hands its dK^T/dV^T partials to pair 0 through LDS: dV in ring0,
  // dK in ring1, each [half][tile][register][lane] fp32 (16 KB)
  float* partv = reinterpret_cast<float*>(ring);
  float* partk = reinterpret_cast<float*>(ring + ENTRY);
  __syncthreads();
  auto slot = [&](int which, int i) {
    return (which < 2 ? partv : partk) + ((half * 2 + (which & 1)) * 16 + i) * 64 + lane;
  };
  if (pair == 1) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      *slot(0, i) = dv0[i];
      *slot(1, i) = dv1[i];
      *slot(2, i) = dk0[i];
      *slot(3, i) = dk1[i];
    }
  }
  __syncthreads();
  if (pair == 0) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      dv0[i] += *slot(0, i);
      dv1[i] += *slot(1, i);
      dk0[i] += *slot(2, i);
      dk1[i] += *slot(3, i);
    }
    // accumulators are transposed: lane holds key kr, d = 32*dt + 8*g + 4*hh + 0..3
    const float as = p.attn_scale;
    T* dkr = dk + kr * kD;
    T* dvr = dv + kr * kD;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      store4(dvr + 8 * g + 4 * hh, dv0[4 * g], dv0[4 * g + 1], dv0[4 * g + 2], dv0[4 * g + 3]);
      store4(dvr + 32 + 8 * g + 4 * hh, dv1[4 * g], dv1[4 * g + 1], dv1[4 * g + 2], dv1[4 * g + 3]);
      store4(dkr + 8 * g + 4 * hh, as * dk0[4 * g], as * dk0[4 * g + 1], as * dk0[4 * g + 2],
             as * dk0[4 * g + 3]);
      store4(dkr + 32 + 8 * g + 4 * hh, as * dk1[4 * g], as * dk1[4 * g + 1], as * dk1[4 * g + 2],
             as * dk1[4 * g + 3]);
    }
  }
}

// -------------------------------------- score and landmark gradients ----

// dsel[t, s] = w_s (dw_s - sum_s' w_s' dw_s'), dw summed over the group's heads.
__global__ __launch_bounds__(64) void dsel_kernel(const float* __restrict__ w, const float* __restrict__ dwp,
                                                  float* __restrict__ dsel, int64_t nQ, int H, int Hr, int K,
                                                  int causal) {
  const int64_t row = blockIdx.x;  // (b, hr, t)
  const int64_t t = row % nQ;
  const int64_t bhr = row / nQ;
  const int64_t b = bhr / Hr;
  const int hr = (int)(bhr % Hr);
  const int s = threadIdx.x;
  float dw = 0.f, ws = 0.f;
  if (s < K) {
    ws = w[row * K + s];
    if (t + causal < nQ) {
      const int h0 = Hr == 1 ? 0 : hr, h1 = Hr == 1 ? H : hr + 1;
      for (int h = h0; h < h1; ++h) dw += dwp[((b * H + h) * nQ + t) * K + s];
    }
  }
  float tot = ws * dw;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) tot += __shfl_xor(tot, o);
  if (s < K) dsel[row * K + s] = ws * (dw - tot);
}

// dlmk_q[t] = score_scale * sum_s dsel[t, s] lmk_k[idx[t, s]]
template <typename T>
__global__ __launch_bounds__(256) void dlmk_q_kernel(const T* __restrict__ lk, const int32_t* __restrict__ idx,
                                                     const float* __restrict__ dsel, float* __restrict__ dlq,
                                                     int64_t nQ, int64_t nKV, int D, int K, float scale) {
  const int64_t row = blockIdx.x;
  const int64_t bhr = row / nQ;
  for (int x = threadIdx.x; x < D; x += 256) {
    float acc = 0.f;
    for (int s = 0; s < K; ++s) {
      const int j = idx[row * K + s];
      if (j >= 0 && j < nKV) acc += dsel[row * K + s] * to_f32(lk[(bhr * nKV + j) * D + x]);
    }
    dlq[row * D + x] = scale * acc;
  }
}

// dlmk_k[j] = score_scale * sum over the rows (t, s) that retrieved j of dsel[t, s] lmk_q[t]
template <typename T>
__global__ __launch_bounds__(256) void dlmk_k_kernel(const T* __restrict__ lq, const int* __restrict__ offs,
                                                     const int* __restrict__ sorted, const float* __restrict__ dsel,
                                                     float* __restrict__ dlk, int64_t nQ, int64_t nKV, int D, int K,
                                                     float scale) {
  const int64_t wid = blockIdx.x;  // (b, hr, j)
  const int64_t bhr = wid / nKV, j = wid % nKV;
  const int* off = offs + bhr * (nKV + 1);
  const int lo = off[j], hi = off[j + 1];
  const int* list = sorted + bhr * nQ * K;
  for (int x = threadIdx.x; x < D; x += 256) {
    float acc = 0.f;
    for (int u = lo; u < hi; ++u) {
      const int e = list[u];
      const int64_t t = e / K;
      acc += dsel[(bhr * nQ) * K + e] * to_f32(lq[(bhr * nQ + t) * D + x]);
    }
    dlk[wid * D + x] = scale * acc;
  }
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

template <typename T>
hipError_t launch_bwd_t(const Shape& s, BwdParams& p, float* dsel, const void* lmk_q, const void* lmk_k,
                        float* dlmk_q, float* dlmk_k, hipStream_t st) {
  const int64_t BHr = (int64_t)s.B * s.Hr, BH = (int64_t)s.B * s.H;
  const int64_t nent = BHr * s.nQ * s.topk;
  Ws& w = p.ws;
  hipLaunchKernelGGL(weights_kernel, dim3(blocks_for(nent, 256)), dim3(256), 0, st, p.idx, p.sel, w.w,
                     BHr * s.nQ, s.topk, s.nKV);
  note_launch("weights_kernel", st);
  const unsigned zblocks = std::min(blocks_for(BHr * s.nKV, 256), 4096u);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(zblocks), dim3(256), 0, st, w.counts, BHr * s.nKV);
  note_launch("fill_zero_kernel", st);
  hipLaunchKernelGGL(csr_count_kernel, dim3(blocks_for(nent, 256)), dim3(256), 0, st, p.idx, w.counts, BHr, s.nQ,
                     s.topk, s.nKV, s.causal);
  note_launch("csr_count_kernel", st);
  hipLaunchKernelGGL(csr_scan_kernel, dim3((unsigned)BHr), dim3(1024), 0, st, w.counts, w.offs, w.cursor, s.nKV);
  note_launch("csr_scan_kernel", st);
  hipLaunchKernelGGL(csr_fill_kernel, dim3(blocks_for(nent, 256)), dim3(256), 0, st, p.idx, w.cursor, w.unsorted,
                     BHr, s.nQ, s.topk, s.nKV, s.causal);
  note_launch("csr_fill_kernel", st);
  hipLaunchKernelGGL(csr_sort_kernel, dim3(blocks_for(BHr * s.nKV, 4)), dim3(256), 0, st, w.offs, w.unsorted,
                     w.sorted, BHr, s.nQ, s.topk, s.nKV);
  note_launch("csr_sort_kernel", st);
  const int64_t nq_work = BH * s.nQ, nk_work = BH * s.nKV;
  hipLaunchKernelGGL(bwd_dq_kernel<T>, dim3((unsigned)round8(nq_work)), dim3(kThreads), 0, st, p, nq_work);
  note_launch("bwd_dq_kernel", st);
  hipLaunchKernelGGL(bwd_dkdv_kernel<T>, dim3((unsigned)round8(nk_work)), dim3(kThreads), 0, st, p, nk_work);
  note_launch("bwd_dkdv_kernel", st);
  hipLaunchKernelGGL(dsel_kernel, dim3((unsigned)(BHr * s.nQ)), dim3(64), 0, st, w.w, w.dwp, dsel, s.nQ, s.H, s.Hr,
                     s.topk, s.causal);
  note_launch("dsel_kernel", st);
  if (dlmk_q) {
    hipLaunchKernelGGL(dlmk_q_kernel<T>, dim3((unsigned)(BHr * s.nQ)), dim3(256), 0, st, (const T*)lmk_k, p.idx,
                       dsel, dlmk_q, s.nQ, s.nKV, s.D, s.topk, s.score_scale);
    note_launch("dlmk_q_kernel", st);
  }
  if (dlmk_k) {
    hipLaunchKernelGGL(dlmk_k_kernel<T>, dim3((unsigned)(BHr * s.nKV)), dim3(256), 0, st, (const T*)lmk_q, w.offs,
                       w.sorted, dsel, dlmk_k, s.nQ, s.nKV, s.D, s.topk, s.score_scale);
    note_launch("dlmk_k_kernel", st);
  }
  return take_launch_error();
}

}  // namespace

size_t bwd_workspace(const Shape& s) { return carve_size(s); }

hipError_t launch_xattn_bwd(const Shape& s, const void* q, const void* k, const void* v, const int32_t* idx,
                            const float* sel, const float* lse, const void* dout, void* dq, void* dk, void* dv,
                            float* dsel, const void* lmk_q, const void* lmk_k, float* dlmk_q, float* dlmk_k,
                            void* ws, hipStream_t stream) {
  BwdParams p;
  p.q = q; p.k = k; p.v = v; p.idx = idx; p.sel = sel; p.lse = lse; p.dout = dout;
  p.dq = dq; p.dk = dk; p.dv = dv;
  p.ws = carve(s, ws);
  p.B = s.B; p.H = s.H; p.Hr = s.Hr; p.K = s.topk;
  p.nQ = s.nQ; p.nKV = s.nKV;
  p.causal = s.causal;
  p.attn_scale = s.attn_scale;
  return s.bf16 ? launch_bwd_t<__bf16>(s, p, dsel, lmk_q, lmk_k, dlmk_q, dlmk_k, stream)
                : launch_bwd_t<float>(s, p, dsel, lmk_q, lmk_k, dlmk_q, dlmk_k, stream);
}

}  // namespace gca
