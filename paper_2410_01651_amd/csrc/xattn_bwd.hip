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
// With an LMK row per chunk (S + 1 query rows against S-row key chunks) the
// 65th row takes the same steps as a vector against the tiles the waves hold:
// in the query-stationary pass one wave per slot (alternating) forms its
// scores, dP, D and dS with one key per lane and accumulates its dQ row, and
// in the key-stationary pass every wave adds the row's rank-one terms to dV and
// dK with one more, mostly zero, 16-deep MFMA step.
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

// query-stationary pass: wave pairs per workgroup (one, so that a round's
// barrier couples only the two waves sharing a ring), four workgroups per CU
constexpr int kPairs = 1;
constexpr int kThreads = 128 * kPairs;
constexpr int kWgPerCu = 4 / kPairs;

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
  BwdWs ws;
  int B, H, Hr, K;
  int64_t nQ, nKV;
  int causal;
  float attn_scale;
  bool windows;  // dQ stream order (StreamOrder), the forward's
};

// the LMK row's per-chunk exchange between the two waves of a dQ pair
template <typename T>
struct LmkShared {
  T q[2][kD];      // the row's Q and dO, by chunk parity
  T d[2][kD];
  T p[2][kS];      // per wave: the current slot's dS (one per key)
  float o[2][kD];  // per wave: its slots' share of the row's dQ
  float dl[2][32]; // per slot: -D and the shifted lse of the row
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
                                                       int* __restrict__ sorted, int* __restrict__ head, int64_t BHr,
                                                       int64_t nQ, int K, int64_t nKV) {
  const int64_t wv = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wv >= BHr * nKV) return;
  const int lane = threadIdx.x & 63;
  const int64_t bhr = wv / nKV, j = wv % nKV;
  const int* off = offs + bhr * (nKV + 1);
  const int lo = off[j], hi = off[j + 1];
  const int* src = unsorted + bhr * nQ * K;
  int* dst = sorted + bhr * nQ * K;
  int* hd = head + wv * kHeadInts;
  if (lane == 0) {
    hd[0] = lo;
    hd[1] = hi - lo;
  }
  for (int i = lo + lane; i < hi; i += 64) {
    const int e = src[i];
    int rank = 0;
    for (int u = lo; u < hi; ++u) rank += src[u] < e ? 1 : 0;
    dst[lo + rank] = e;
    if (rank < kHeadEntries) hd[2 + rank] = e;
  }
}

// ------------------------------------------------- query-stationary dQ ----

// Persistent workgroups of one wave pair, four per CU; each pair is a stream of
// (batch, head, query chunk) items, taking the chunk's retrieved chunks one per round
// from its two LDS ring slots (K_j and V_j tiles, copied one round ahead), each
// wave owning 32 query tokens.  Per retrieved chunk it writes D_s and the
// shifted log-sum-exp used by the key-stationary pass, and the wave's partial
// sum of D_s for dw; dQ stays in registers until the chunk ends.  The work order
// is the forward's (StreamOrder, chosen the same way).
// STAGE (k <= kDqStageK): the per-(token, slot) values are staged in LDS and
// stored once per chunk.
constexpr int kDqStageK = 8;
template <typename T, bool STAGE, bool XR>
__global__ __launch_bounds__(kThreads, kWgPerCu) void bwd_dq_kernel(BwdParams p, int64_t nwork) {
  constexpr int TILE = kS * kD;
  constexpr int SQ = XR ? kS + 1 : kS;  // query rows per chunk
  static_assert(kPairs == 1, "the LMK row exchange assumes one pair per workgroup");
  __shared__ __attribute__((aligned(16))) LmkShared<T> sX[1];  // used with XR only
  __shared__ __attribute__((aligned(16))) T ring[kPairs * 2 * 2 * TILE];  // pair p: slots 2p, 2p+1
  __shared__ int sJ[kPairs][2][32];     // [pair][chunk parity][slot]: chunk index or -1
  __shared__ int sSlot[kPairs][2][32];  // compacted valid slots: slot, chunk, weight
  __shared__ int sJc[kPairs][2][32];
  __shared__ float sWc[kPairs][2][32];
  __shared__ int sN[kPairs][2];
  // per wave, the (-D, shifted lse) pairs of its 32 tokens x k slots and its dw
  // partials (k <= 8), stored at the end of the chunk: a store still in flight
  // holds up the next round's wait for its copies, so none is issued per round
  constexpr int kStageK = STAGE ? kDqStageK : 1;
  __shared__ float sDL[2 * kPairs][2][kStageK][32];
  __shared__ float sDw[2 * kPairs][kStageK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5;
  const int pair = wave >> 1, half = wave & 1;
  const int xcd = (int)(blockIdx.x & 7);
  const int64_t st_wg = (int64_t)(blockIdx.x >> 3) * kPairs;
  auto order_of = [&](int q) {
    return StreamOrder((int64_t)(gridDim.x >> 3) * kPairs, st_wg + q, xcd, nwork, p.windows);
  };
  const StreamOrder ord = order_of(pair);
  const int64_t my_n = ord.length();
  int64_t nch = 0;  // all pairs of the workgroup run nch chunks of rounds
  for (int q = 0; q < kPairs; ++q) nch = max(nch, order_of(q).length());
  if (nch == 0) return;
  const int64_t c_begin = ord.item(0);
  const int K = p.K;
  const int qi = 32 * half + (lane & 31);
  const int l32 = lane & 31;
  const float sc = p.attn_scale * kLog2e;
  const int cb = 16 * ((lane >> 4) & 1);

  // retrieval row t of a chunk: its offset in idx / w, or -1
  auto row_off_of = [&](const Geo& g) -> int64_t {
    const int hr = p.Hr == 1 ? 0 : g.h;
    const int64_t t = p.causal ? g.c - 1 : 0;
    return t >= 0 ? ((g.b * p.Hr + hr) * p.nQ + t) * K : -1;
  };
  struct Meta {
    int j;
    float w;
  };
  auto load_meta = [&](const Geo& g) -> Meta {
    Meta m{-1, 0.f};
    const int64_t ro = row_off_of(g);
    if (ro >= 0 && lane < K) {
      m.j = p.idx[ro + lane];
      m.w = p.ws.w[ro + lane];
    }
    return m;
  };
  // first wave of a pair: the pair's compacted slot list of a chunk
  auto make_slots = [&](const Meta& m, int buf) __device__ {
    const bool valid = lane < K && m.j >= 0 && m.j < p.nKV;
    const uint64_t mask = __ballot(valid);
    if (lane < 32) sJ[pair][buf][lane] = valid ? m.j : -1;
    if (valid) {
      const int rk = lanes_below(mask);
      sSlot[pair][buf][rk] = lane;
      sJc[pair][buf][rk] = m.j;
      sWc[pair][buf][rk] = m.w;
    }
    if (lane == 0) sN[pair][buf] = __popcll(mask);
  };
  auto tok_of = [&](const Geo& g) -> int64_t { return ((g.b * p.H + g.h) * p.nQ + g.c) * SQ; };
  const int64_t lq_len = p.nQ * SQ;  // query tokens per (batch, head)
  // the LMK row's Q and dO rows: copied straight into LDS (wave 0 the Q row, wave
  // 1 the dO row, one 16-byte piece per lane below kXPieces) with the chunk's
  // Q/dO fragment loads; visible to both waves after the next wait and barrier
  constexpr int kXPieces = kD * (int)sizeof(T) / 16;
  const int xh = __builtin_amdgcn_readfirstlane(half);  // the wave's half, in a scalar register

  // ---- prologue
  Frag<T> qf[4], df[4];  // the current chunk's Q and dO rows of this lane's query
  Meta meta{-1, 0.f};
  Geo g0(c_begin, p.nQ, p.H);
  Geo g1 = g0, g2 = g0;  // (the range order steps without divisions)
  if (p.windows) {
    g1 = Geo(ord.item(1), p.nQ, p.H);
    g2 = Geo(ord.item(2), p.nQ, p.H);
  } else {
    g1.next(p.nQ, p.H, ord.S);
    g2 = g1;
    g2.next(p.nQ, p.H, ord.S);
  }
  auto load_qdo = [&](const Geo& g, Frag<T>* qd, Frag<T>* dd, int xbuf) __device__ {
    const int64_t row = tok_of(g) + (XR ? opaque(qi) : qi);
    const T* qr = reinterpret_cast<const T*>(p.q) + row * kD;
    const T* dr = reinterpret_cast<const T*>(p.dout) + row * kD;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      qd[kb] = load_frag(qr + 16 * kb + 8 * hh);
      dd[kb] = load_frag(dr + 16 * kb + 8 * hh);
    }
    if (XR && lane < kXPieces) {
      const int64_t xrow = (tok_of(g) + kS) * kD;
      const T* src = reinterpret_cast<const T*>(xh == 0 ? p.q : p.dout) + xrow;
      dma_row16(src, lane * 16u, xh == 0 ? &sX[0].q[xbuf][0] : &sX[0].d[xbuf][0]);
    }
  };
  if (my_n > 0) {
    const Meta m0 = load_meta(g0);
    load_qdo(g0, qf, df, 0);
    if (half == 0) make_slots(m0, 0);
    if (my_n > 1) meta = load_meta(g1);
  }
  wait_vmem<0>();
  __syncthreads();

  const TileCopy<T, 2> cp(half, lane);
  const T* const gk = reinterpret_cast<const T*>(p.k);
  const T* const gv = reinterpret_cast<const T*>(p.v);
  auto slice_of = [&](const Geo& g) __device__ { return (g.b * p.H + g.h) * p.nKV * TILE; };
  auto issue_item = [&](int64_t kvb, int j, int slot) __device__ {
    j = min(max(j, 0), (int)p.nKV - 1);  // lists hold valid chunks; never copy from outside the slice
    T* dst = ring + (2 * pair + slot) * (2 * TILE);
    cp.issue(gk + kvb + (int64_t)j * TILE, dst);
    cp.issue(gv + kvb + (int64_t)j * TILE, dst + TILE);
  };
  int ls = sSlot[pair][0][l32], lj = sJc[pair][0][l32];
  float lw = sWc[pair][0][l32];
  int64_t kvb = uniform64(slice_of(g0)), kvb_n = 0;
  int cs = 0;
  // this lane's saved lse of the next item to compute (loaded a round ahead),
  // and the LMK row's
  float lse_next = 0.f, lsex_next = 0.f;
  if (my_n > 0 && sN[pair][0] > 0) {
    issue_item(kvb, __builtin_amdgcn_readlane(lj, 0), cs);
    lse_next = p.lse[(tok_of(g0) + qi) * K + __builtin_amdgcn_readlane(ls, 0)];
    if (XR) lsex_next = p.lse[(tok_of(g0) + kS) * K + __builtin_amdgcn_readlane(ls, 0)];
  }

  constexpr bool kB16 = std::is_same<T, __bf16>::value;
  constexpr uint32_t kTileB = TILE * sizeof(T), kRowB = kD * sizeof(T);
  const lds_char* const lds0 = (const lds_char*)(ring);
  uint32_t kofs[4], tofs[2][2];
  {
    const uint32_t pb = (uint32_t)pair * 4 * kTileB;
    const int s16 = lane & 15;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) kofs[kb] = pb + Swz<T>::off(lane & 31, 16 * kb + 8 * hh) * sizeof(T);
#pragma unroll
    for (int dh = 0; dh < 2; ++dh)
#pragma unroll
      for (int r8 = 0; r8 < 2; ++r8)
        tofs[dh][r8] = pb + Swz<T>::off(8 * r8 + 4 * hh + (s16 >> 2), 32 * dh + cb + 4 * (s16 & 3)) * sizeof(T);
  }

  f32x16 g0a = zero16(), g1a = zero16();  // dQ^T, d rows 0-31 / 32-63
  // cbase: element of (this slice, slot 0, this chunk's first token) in Dbuf / Lbuf
  // pre: this is the chunk's last item and a next chunk follows; its Q and dO rows
  // are loaded as soon as this item's products have read qf/df, so that the
  // next chunk's first round does not wait out the whole load
  float ox0 = 0.f, ox1 = 0.f;  // LMK row: this lane's partial dQ for d = l%32 and 32 + l%32
  auto run = [&](int slot, int u, float lse_q, float lse_x, int64_t cbase, int64_t t, bool pre, int buf) __device__ {
    const uint32_t co = (uint32_t)slot * 2 * kTileB;
    // With the LMK row every register counts: the other fragment offsets are
    // derived from the first two each round by their swizzle's fixed XOR
    // patterns (key block kb: bits 5-6; transposed halves: bit 6, and rows +8:
    // bits 4 and 10), instead of being held across the whole loop.
    uint32_t k0b = kofs[0], t0b = tofs[0][0];
    if constexpr (XR && kB16) {
      k0b = (uint32_t)opaque((int)k0b);
      t0b = (uint32_t)opaque((int)t0b);
    }
    auto KO = [&](int kb) -> uint32_t { return (XR && kB16) ? (k0b ^ (uint32_t)(kb << 5)) : kofs[kb]; };
    auto TO = [&](int dh, int r8) -> uint32_t {
      return (XR && kB16) ? (t0b ^ (uint32_t)((dh << 6) | (r8 ? 1040 : 0))) : tofs[dh][r8];
    };
    const int s = __builtin_amdgcn_readlane(ls, u);
    const float ws = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lw), u));
    const bool xr = XR && (u & 1) == xh;  // this wave takes the LMK row of slot u
    const T* sK = ring + (2 * pair + slot) * (2 * TILE);
    const T* sV = sK + TILE;
    // the LMK row: scores and dP with one key per lane (row fragments of K and V
    // against the row's Q and dO, the two dimension halves added across l ^ 32),
    // w P, D, dS, and its dQ against the K^T fragments
    float Dx = 0.f;
    if (xr) {
      __builtin_amdgcn_sched_barrier(0);  // the row's reads start after the tile's products
      float a0 = 0.f, a1 = 0.f, b0 = 0.f, b1 = 0.f;
#pragma unroll
      for (int kb = 0; kb < 8; ++kb) {
        __builtin_amdgcn_sched_barrier(0);  // one key block's fragments live at a time
        const int kk = kb & 3;
        const bool vt = kb >= 4;  // blocks 0-3: K against the row's Q; 4-7: V against its dO
        const Frag<T> xv = vec_frag(vt ? &sX[0].d[buf][0] : &sX[0].q[buf][0], 16 * kk + 8 * hh);
        Frag<T> r0, r1;
        if constexpr (kB16) {
          const lds_char* kp = lds0 + (KO(kk) + co) + (vt ? kTileB : 0u);
          r0 = lds_b128_at(kp);
          r1 = lds_b128_at(kp + 32 * kRowB);
        } else {
          r0 = lds_frag(vt ? sV : sK, lane & 31, 16 * kk + 8 * hh);
          r1 = lds_frag(vt ? sV : sK, 32 + (lane & 31), 16 * kk + 8 * hh);
        }
        if (vt) {
          b0 = frag_dot(r0, xv, b0);
          b1 = frag_dot(r1, xv, b1);
        } else {
          a0 = frag_dot(r0, xv, a0);
          a1 = frag_dot(r1, xv, a1);
        }
      }
      a0 = sum_xor32(a0);
      a1 = sum_xor32(a1);
      b0 = sum_xor32(b0);
      b1 = sum_xor32(b1);
      const float xs = hh ? a1 : a0, xdp = hh ? b1 : b0;  // key `lane`
      const float wsf = fmaxf(ws, 1e-30f);
      const float offx = lse_x * kLog2e - __builtin_amdgcn_logf(wsf);
      const float wpx = __builtin_amdgcn_exp2f(fmaf(xs, sc, -offx));
      Dx = sum64(wpx * xdp) * __builtin_amdgcn_rcpf(wsf);
      sX[0].p[xh][lane] = (T)(wpx * (xdp - Dx));
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        __builtin_amdgcn_sched_barrier(0);  // one key block's fragments live at a time
        Frag<T> k0, k1;
        if constexpr (kB16) {
          k0 = lds_tr2(lds0 + (TO(0, 0) + co) + 16 * kb * kRowB, lds0 + (TO(0, 1) + co) + 16 * kb * kRowB);
          k1 = lds_tr2(lds0 + (TO(1, 0) + co) + 16 * kb * kRowB, lds0 + (TO(1, 1) + co) + 16 * kb * kRowB);
        } else {
          k0 = lds_frag_t(sK, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb);
          k1 = lds_frag_t(sK, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb);
        }
        const Frag<T> xf = vec_frag_t(&sX[0].p[xh][0], 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh);
        ox0 = frag_dot(k0, xf, ox0);
        ox1 = frag_dot(k1, xf, ox1);
      }
      if (lane == 0) {
        sX[0].dl[0][s] = -Dx;
        sX[0].dl[1][s] = lse_x * kLog2e - __builtin_amdgcn_logf(ws);
      }
      __builtin_amdgcn_sched_barrier(0);  // the tile's own products start after the row's
    }
    f32x16 s0 = zero16(), s1 = zero16(), p0 = zero16(), p1 = zero16();
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      if constexpr (kB16) {
        const lds_char* kp = lds0 + (KO(kb) + co);
        mma32(s0, lds_b128_at(kp), qf[kb]);
        mma32(s1, lds_b128_at(kp + 32 * kRowB), qf[kb]);
        mma32(p0, lds_b128_at(kp + kTileB), df[kb]);
        mma32(p1, lds_b128_at(kp + (kTileB + 32 * kRowB)), df[kb]);
      } else {
        mma32(s0, lds_frag(sK, lane & 31, 16 * kb + 8 * hh), qf[kb]);
        mma32(s1, lds_frag(sK, 32 + (lane & 31), 16 * kb + 8 * hh), qf[kb]);
        mma32(p0, lds_frag(sV, lane & 31, 16 * kb + 8 * hh), df[kb]);
        mma32(p1, lds_frag(sV, 32 + (lane & 31), 16 * kb + 8 * hh), df[kb]);
      }
    }
    if (pre) load_qdo(g1, qf, df, buf ^ 1);
    // w P^T (the weight folded into the exponent: wsf = max(ws, 1e-30) keeps the
    // shift finite), D = rowsum(P o dP) for this lane's query, w dS
    const float wsf = fmaxf(ws, 1e-30f);
    const float off = lse_q * kLog2e - __builtin_amdgcn_logf(wsf);
    float Dw = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      s0[i] = __builtin_amdgcn_exp2f(fmaf(s0[i], sc, -off));
      s1[i] = __builtin_amdgcn_exp2f(fmaf(s1[i], sc, -off));
      Dw = fmaf(s0[i], p0[i], Dw);
      Dw = fmaf(s1[i], p1[i], Dw);
    }
    const float Dq = sum_xor32(Dw) * __builtin_amdgcn_rcpf(wsf);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      s0[i] = s0[i] * (p0[i] - Dq);
      s1[i] = s1[i] * (p1[i] - Dq);
    }
    Frag<T> f[4];
    frag_from_acc(f[0], s0, 0, 1.f);
    frag_from_acc(f[1], s0, 1, 1.f);
    frag_from_acc(f[2], s1, 0, 1.f);
    frag_from_acc(f[3], s1, 1, 1.f);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      if constexpr (kB16) {
        mma32(g0a, lds_tr2(lds0 + (TO(0, 0) + co) + 16 * kb * kRowB, lds0 + (TO(0, 1) + co) + 16 * kb * kRowB),
              f[kb]);
        mma32(g1a, lds_tr2(lds0 + (TO(1, 0) + co) + 16 * kb * kRowB, lds0 + (TO(1, 1) + co) + 16 * kb * kRowB),
              f[kb]);
      } else {
        mma32(g0a, lds_frag_t(sK, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb), f[kb]);
        mma32(g1a, lds_frag_t(sK, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb), f[kb]);
      }
    }
    // D_s (negated: it seeds the dP accumulator there) and the shifted lse of this
    // (query, slot) for the key-stationary pass
    if (hh == 0) {
      const float dneg = -Dq, lsh = lse_q * kLog2e - __builtin_amdgcn_logf(ws);
      if constexpr (STAGE) {
        sDL[wave][0][s][l32] = dneg;
        sDL[wave][1][s][l32] = lsh;
      } else {
        const int64_t o = cbase + s * lq_len + (XR ? opaque(qi) : qi);
        p.ws.Dbuf[o] = dneg;
        p.ws.Lbuf[o] = lsh;
      }
    }
    // this wave's 32 queries' share of dw[t, s] (and the LMK row's D)
    const float dsum = sum32(Dq) + Dx;
    if (lane == 0) {
      if constexpr (STAGE) sDw[wave][s] = dsum;
      else p.ws.dwp[(t * K + s) * 2 + half] = dsum;
    }
  };

  for (int64_t ci = 0; ci < nch; ++ci) {
    const bool live = ci < my_n, live_next = ci + 1 < my_n;
    const int buf = (int)(ci & 1);
    const int n = live ? sN[pair][buf] : 0;
    const int64_t tok0 = tok_of(g0);
    const int64_t cbase = (g0.b * p.H + g0.h) * K * lq_len + g0.c * SQ;
    const int64_t tglob = (g0.b * p.H + g0.h) * p.nQ + (p.causal ? g0.c - 1 : 0);  // dw row (b, h, t)
    const int64_t tok_n = tok_of(g1);
    for (int u = 0; u < K; ++u) {
      wait_vmem<0>();
      block_barrier();
      if (u == 0) {
        if (ci > 0 && live) {
          ls = sSlot[pair][buf][l32];
          lj = sJc[pair][buf][l32];
          lw = sWc[pair][buf][l32];
          kvb = kvb_n;
        }
        if (live_next) {
          if (half == 0) make_slots(meta, buf ^ 1);
          if (ci + 2 < my_n) meta = load_meta(g2);
          kvb_n = uniform64(slice_of(g1));
        }
        if (K == 1) block_barrier();  // the next chunk's list is needed this round
      }
      const bool comp = u < n;
      const int is = comp ? cs ^ 1 : cs;
      const float lse_q = lse_next, lse_x = lsex_next;
      if (u + 1 < n) {
        issue_item(kvb, __builtin_amdgcn_readlane(lj, u + 1), is);
        lse_next = p.lse[(tok0 + (XR ? opaque(qi) : qi)) * K + __builtin_amdgcn_readlane(ls, u + 1)];
        if (XR) lsex_next = p.lse[(tok0 + kS) * K + __builtin_amdgcn_readlane(ls, u + 1)];
      } else if (u == K - 1 && live_next && sN[pair][buf ^ 1] > 0) {
        issue_item(kvb_n, sJc[pair][buf ^ 1][0], is);
        lse_next = p.lse[(tok_n + (XR ? opaque(qi) : qi)) * K + sSlot[pair][buf ^ 1][0]];
        if (XR) lsex_next = p.lse[(tok_n + kS) * K + sSlot[pair][buf ^ 1][0]];
      }
      if (comp) {
        run(cs, u, lse_q, lse_x, cbase, tglob, live_next && u == n - 1, buf);
        cs ^= 1;
      }
      // a chunk without items loads the next chunk's Q and dO rows in its first round
      if (n == 0 && u == 0 && live_next) load_qdo(g1, qf, df, buf ^ 1);
    }

    // ---- finish the chunk: dQ rows of this wave; zero dw partials of empty slots
    if (live) {
      const float as = p.attn_scale;
      T* drow = reinterpret_cast<T*>(p.dq) + (tok0 + (XR ? opaque(qi) : qi)) * kD;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        store4(drow + 8 * g + 4 * hh, as * g0a[4 * g], as * g0a[4 * g + 1], as * g0a[4 * g + 2],
               as * g0a[4 * g + 3]);
        store4(drow + 32 + 8 * g + 4 * hh, as * g1a[4 * g], as * g1a[4 * g + 1], as * g1a[4 * g + 2],
               as * g1a[4 * g + 3]);
      }
      const bool has_row = !p.causal || g0.c > 0;
      if constexpr (XR) {
        // the LMK row: add the two waves' shares of its dQ, store it and its
        // per-slot -D and shifted lse
        const float t0 = sum_xor32(ox0), t1 = sum_xor32(ox1);
        sX[0].o[xh][lane] = hh ? t1 : t0;  // lane l: d = l
        block_barrier();
        if (xh == 0) {
          // (lane-dependent addresses are formed here, not kept in registers
          // across the whole loop)
          const int ln = opaque(lane);
          const int64_t tx = tok0 + kS;
          reinterpret_cast<T*>(p.dq)[tx * kD + ln] = (T)(as * (sX[0].o[0][lane] + sX[0].o[1][lane]));
          if (lane < K && sJ[pair][buf][lane] >= 0) {
            const int64_t o = cbase + ln * lq_len + kS;
            p.ws.Dbuf[o] = sX[0].dl[0][lane];
            p.ws.Lbuf[o] = sX[0].dl[1][lane];
          }
        }
        ox0 = 0.f;
        ox1 = 0.f;
      }
      if constexpr (STAGE) {
        // this wave's staged values (its own LDS writes, read back in program
        // order): per valid slot one contiguous run of 32 tokens
        for (int e = lane; e < 32 * K; e += 64) {
          const int sl = e >> 5, q = e & 31;
          if (sJ[pair][buf][sl] >= 0) {
            const int64_t o = cbase + sl * lq_len + 32 * half + (XR ? opaque(q) : q);
            p.ws.Dbuf[o] = sDL[wave][0][sl][q];
            p.ws.Lbuf[o] = sDL[wave][1][sl][q];
          }
        }
        if (has_row && lane < K) {
          const int sl = opaque(lane);
          p.ws.dwp[(tglob * K + sl) * 2 + xh] = sJ[pair][buf][lane] >= 0 ? sDw[wave][lane] : 0.f;
        }
      } else if (has_row && n < K && lane < K && sJ[pair][buf][lane] < 0) {
        const int sl = opaque(lane);
        p.ws.dwp[(tglob * K + sl) * 2 + xh] = 0.f;
      }
    }
    g0a = zero16();
    g1a = zero16();
    g0 = g1;
    g1 = g2;
    if (p.windows)
      g2 = Geo(ord.item(ci + 3), p.nQ, p.H);
    else
      g2.next(p.nQ, p.H, ord.S);
  }
}

// ---------------------------------------------- key-stationary dK, dV ----

// One workgroup of two waves per (batch, head, key chunk j), four per CU; the pair
// takes the retrievers (row t, slot s) of chunk j in list order through a
// two-slot LDS ring (Q_c and dO_c tiles plus the shifted-lse and D columns of
// slot s, which the query-stationary pass wrote), each wave owning 32 of chunk
// j's keys, so a workgroup's barrier couples only its two waves and no partial
// sums are exchanged.  With the shifted lse L = log2(e) lse - log2(w_s),
// exp2(S log2(e) scale - L) is w_s P_s directly.
constexpr int kKvThreads = 128;
template <typename T, bool XR>
__global__ __launch_bounds__(kKvThreads, 4) void bwd_dkdv_kernel(BwdParams p, int64_t nwork) {
  constexpr int TILE = kS * kD;
  constexpr int SQ = XR ? kS + 1 : kS;  // query rows per chunk
  // ring slot: Q_c tile, dO_c tile, shifted-lse column, D column; with the LMK
  // row also its Q and dO rows and its shifted lse and -D (16 bytes)
  constexpr int XOFF = 2 * TILE + 2 * kS * (int)(sizeof(float) / sizeof(T));
  constexpr int ENTRY = XOFF + (XR ? 2 * kD + 16 / (int)sizeof(T) : 0);
  __shared__ __attribute__((aligned(16))) T ring[2 * ENTRY];
  constexpr int NE = 256;  // retrievers staged in LDS per batch
  __shared__ int sE[NE];
  // LMK rows: up to kXGroup retrievers' rows staged for one padded contraction
  // step: Q and dO rows transposed ([d][retriever]) and, per key, w P and dS
  // ([key][retriever])
  constexpr int kXGroup = 8;
  __shared__ __attribute__((aligned(16))) T sXst[XR ? 4 : 1][XR ? kD : 1][kXGroup];

  const int64_t wid = xcd_swizzle(blockIdx.x, gridDim.x);
  if (wid >= nwork) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5;
  const int half = wave;
  const int64_t j = wid % p.nKV;
  const int64_t bh = wid / p.nKV;
  const int h = (int)(bh % p.H);
  const int64_t b = bh / p.H;
  const int hr = p.Hr == 1 ? 0 : h;
  const int K = p.K;
  const int64_t bhr = b * p.Hr + hr;
  // the chunk's header row: lane i < kHeadInts holds int i
  const int hv = lane < kHeadInts ? p.ws.head[(bhr * p.nKV + j) * kHeadInts + lane] : 0;
  const int lo = __builtin_amdgcn_readlane(hv, 0), n = __builtin_amdgcn_readlane(hv, 1);
  const int* list_g = p.ws.sorted + bhr * p.nQ * K + lo;

  const int64_t key0 = (bh * p.nKV + j) * kS;  // first key token of chunk j
  T* dk = reinterpret_cast<T*>(p.dk) + key0 * kD;
  T* dv = reinterpret_cast<T*>(p.dv) + key0 * kD;
  if (n == 0) {
    for (int e = tid; e < kS * kD / 4; e += kKvThreads) {
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

  const int64_t lq_len = p.nQ * SQ;  // query tokens per (batch, head)
  const T* qb = reinterpret_cast<const T*>(p.q) + bh * lq_len * kD;
  const T* ob = reinterpret_cast<const T*>(p.dout) + bh * lq_len * kD;
  const float* Lb = p.ws.Lbuf + bh * lq_len * K;
  const float* Db = p.ws.Dbuf + bh * lq_len * K;

  const TileCopy<T, 2> cp(wave, lane);
  const uint32_t col_off = (uint32_t)(lane * sizeof(float));
  constexpr int kXPieces = kD * (int)sizeof(T) / 16;  // 16-byte pieces of one row
  const int xw = __builtin_amdgcn_readfirstlane(wave);  // LMK row copies: wave 0 Q and L, wave 1 dO and -D
  const T* const xrow_src = xw == 0 ? qb : ob;
  const float* const xcol_src = xw == 0 ? Lb : Db;
  auto enc = [&](int e) { return ((e / K + p.causal) << 5) | (e % K); };  // list entry t*K+s -> (query chunk << 5) | slot
  auto issue = [&](int slot, int cs) __device__ {
    const int64_t c = cs >> 5;
    const int s = cs & 31;
    T* dst = ring + slot * ENTRY;
    cp.issue(qb + c * SQ * kD, dst);
    cp.issue(ob + c * SQ * kD, dst + TILE);
    float* cols = reinterpret_cast<float*>(dst + 2 * TILE);
    if (wave == 0) dma_column_s(Lb + s * lq_len + c * SQ, col_off, cols);
    else dma_column_s(Db + s * lq_len + c * SQ, col_off, cols + kS);
    if constexpr (XR) {
      // the LMK row (row S of the chunk): wave 0 its Q row and shifted lse, wave 1
      // its dO row and -D (addresses in scalar registers)
      const int64_t xr = c * SQ + kS;
      T* xdst = dst + XOFF;
      float* xcol = reinterpret_cast<float*>(xdst + 2 * kD);
      if (lane < kXPieces) dma_row16(xrow_src + xr * kD, lane * 16u, xdst + xw * kD);
      if (lane == 0) dma_column_s(xcol_src + s * lq_len + xr, 0u, xcol + xw);
    }
  };

  f32x16 dv0 = zero16(), dv1 = zero16(), dk0 = zero16(), dk1 = zero16();
  const float sc = p.attn_scale * kLog2e;
  const int cb = 16 * ((lane >> 4) & 1);

  // bf16 fragment addresses: this lane's byte offsets inside a ring slot, computed
  // once; a round adds its slot's offset and every fragment read is one of these
  // addresses plus an immediate (row +32, key block, dO tile, transposed-row gap)
  constexpr bool kB16 = std::is_same<T, __bf16>::value;
  constexpr uint32_t kTileB = TILE * sizeof(T), kRowB = kD * sizeof(T), kEntryB = ENTRY * sizeof(T);
  const lds_char* const lds0 = (const lds_char*)(ring);
  uint32_t rofs[4], tofs[2][2];
  {
    const int s16 = lane & 15;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) rofs[kb] = Swz<T>::off(lane & 31, 16 * kb + 8 * hh) * sizeof(T);
#pragma unroll
    for (int dh = 0; dh < 2; ++dh)
#pragma unroll
      for (int r8 = 0; r8 < 2; ++r8)
        tofs[dh][r8] = Swz<T>::off(8 * r8 + 4 * hh + (s16 >> 2), 32 * dh + cb + 4 * (s16 & 3)) * sizeof(T);
  }
  auto row_frag = [&](const T* tile, uint32_t so, int kb, int half32) __device__ -> Frag<T> {
    if constexpr (kB16) {
      return lds_b128_at(lds0 + (rofs[kb] + so) + half32 * 32 * kRowB);
    } else {
      return lds_frag(tile, 32 * half32 + (lane & 31), 16 * kb + 8 * hh);
    }
  };
  auto col_frag = [&](const T* tile, uint32_t so, int kb, int dh) __device__ -> Frag<T> {
    if constexpr (kB16) {
      return lds_tr2(lds0 + (tofs[dh][0] + so) + 16 * kb * kRowB, lds0 + (tofs[dh][1] + so) + 16 * kb * kRowB);
    } else {
      return lds_frag_t(tile, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 * dh + cb);
    }
  };

  auto run = [&](int slot, int u, bool last) __device__ {
    const T* sQ = ring + slot * ENTRY;
    const T* sO = sQ + TILE;
    const uint32_t qo = (uint32_t)slot * kEntryB, oo = qo + kTileB;
    const float* sL = reinterpret_cast<const float*>(sQ + 2 * TILE);
    const float* sD = sL + kS;
    if constexpr (XR) {
      // with the LMK row the 64 queries go in two halves of 32, one after the
      // other (the same products in the same order per accumulator, half the
      // score and dP registers live at a time)
#pragma unroll
      for (int qh = 0; qh < 2; ++qh) {
        f32x16 pp, ss = zero16();
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 d0 = *reinterpret_cast<const f32x4*>(sD + 32 * qh + 8 * g + 4 * hh);
#pragma unroll
          for (int r = 0; r < 4; ++r) pp[4 * g + r] = d0[r];
        }
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) mma32(ss, row_frag(sQ, qo, kb, qh), kf[kb]);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) mma32(pp, row_frag(sO, oo, kb, qh), vf[kb]);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 l0 = *reinterpret_cast<const f32x4*>(sL + 32 * qh + 8 * g + 4 * hh);
#pragma unroll
          for (int r = 0; r < 4; ++r) ss[4 * g + r] = __builtin_amdgcn_exp2f(fmaf(ss[4 * g + r], sc, -l0[r]));
        }
        Frag<T> wp2[2], ds2[2];
        frag_from_acc(wp2[0], ss, 0, 1.f);
        frag_from_acc(wp2[1], ss, 1, 1.f);
#pragma unroll
        for (int i = 0; i < 16; ++i) pp[i] *= ss[i];
        frag_from_acc(ds2[0], pp, 0, 1.f);
        frag_from_acc(ds2[1], pp, 1, 1.f);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          mma32(dv0, col_frag(sO, oo, 2 * qh + kk, 0), wp2[kk]);
          mma32(dv1, col_frag(sO, oo, 2 * qh + kk, 1), wp2[kk]);
        }
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          mma32(dk0, col_frag(sQ, qo, 2 * qh + kk, 0), ds2[kk]);
          mma32(dk1, col_frag(sQ, qo, 2 * qh + kk, 1), ds2[kk]);
        }
      }
    } else {
      // accumulator row i of a 32-query tile holds query 32*qt + 8*(i/4) + 4*hh + i%4,
      // so four consecutive registers take one 16-byte column read.
      // dP - D = dO V^T + (-D): the accumulators start from the stored -D column
      f32x16 p0, p1;
  #pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 d0 = *reinterpret_cast<const f32x4*>(sD + 8 * g + 4 * hh);
        const f32x4 d1 = *reinterpret_cast<const f32x4*>(sD + 32 + 8 * g + 4 * hh);
  #pragma unroll
        for (int r = 0; r < 4; ++r) {
          p0[4 * g + r] = d0[r];
          p1[4 * g + r] = d1[r];
        }
      }
      // S = Q K^T for this wave's keys (queries 0-31 in s0, 32-63 in s1), and dP
      f32x16 s0 = zero16(), s1 = zero16();
  #pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        mma32(s0, row_frag(sQ, qo, kb, 0), kf[kb]);
        mma32(s1, row_frag(sQ, qo, kb, 1), kf[kb]);
      }
  #pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        mma32(p0, row_frag(sO, oo, kb, 0), vf[kb]);
        mma32(p1, row_frag(sO, oo, kb, 1), vf[kb]);
      }
      // w P (fp32), then dS = w P o (dP - D)
  #pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 l0 = *reinterpret_cast<const f32x4*>(sL + 8 * g + 4 * hh);
        const f32x4 l1 = *reinterpret_cast<const f32x4*>(sL + 32 + 8 * g + 4 * hh);
  #pragma unroll
        for (int r = 0; r < 4; ++r) {
          s0[4 * g + r] = __builtin_amdgcn_exp2f(fmaf(s0[4 * g + r], sc, -l0[r]));
          s1[4 * g + r] = __builtin_amdgcn_exp2f(fmaf(s1[4 * g + r], sc, -l1[r]));
        }
      }
      Frag<T> wp[4], ds[4];
      frag_from_acc(wp[0], s0, 0, 1.f);
      frag_from_acc(wp[1], s0, 1, 1.f);
      frag_from_acc(wp[2], s1, 0, 1.f);
      frag_from_acc(wp[3], s1, 1, 1.f);
  #pragma unroll
      for (int i = 0; i < 16; ++i) {
        p0[i] *= s0[i];
        p1[i] *= s1[i];
      }
      frag_from_acc(ds[0], p0, 0, 1.f);
      frag_from_acc(ds[1], p0, 1, 1.f);
      frag_from_acc(ds[2], p1, 0, 1.f);
      frag_from_acc(ds[3], p1, 1, 1.f);
      // dV^T += dO^T (w P) and dK^T += Q^T dS  (contractions over the 64 queries)
  #pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        mma32(dv0, col_frag(sO, oo, kb, 0), wp[kb]);
        mma32(dv1, col_frag(sO, oo, kb, 1), wp[kb]);
      }
  #pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        mma32(dk0, col_frag(sQ, qo, kb, 0), ds[kb]);
        mma32(dk1, col_frag(sQ, qo, kb, 1), ds[kb]);
      }
    }
    if constexpr (XR) {
      // the LMK row against this wave's keys, after the tile's products (so its
      // registers do not add to theirs): its score and dP for key kr (row
      // fragments of K and V held in registers, the dimension halves added
      // across l ^ 32), w P and dS, staged with the row's Q and dO as retriever
      // u % kXGroup; every kXGroup retrievers (and at the end of a batch) the
      // staged rows enter dV^T += dO_X^T (w P_X) and dK^T += Q_X^T dS_X as one
      // contraction step padded to 16 with zeros
      __builtin_amdgcn_sched_barrier(0);
      const T* sqx = sQ + XOFF;
      const T* sdx = sqx + kD;
      const float* slx = reinterpret_cast<const float*>(sdx + kD);
      float a = 0.f, b = 0.f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        a = frag_dot(kf[kb], vec_frag(sqx, 16 * kb + 8 * hh), a);
        b = frag_dot(vf[kb], vec_frag(sdx, 16 * kb + 8 * hh), b);
      }
      a = sum_xor32(a);
      b = sum_xor32(b);
      const float wpx = __builtin_amdgcn_exp2f(fmaf(a, sc, -slx[0]));
      const float xd = wpx * (b + slx[1]);
      const int e = u % kXGroup;
      if (hh == 0) {
        sXst[2][kr][e] = (T)wpx;
        sXst[3][kr][e] = (T)xd;
      }
      sXst[half][lane][e] = (half == 0 ? sqx : sdx)[lane];  // wave 0 the Q row, wave 1 the dO row
      if (e == kXGroup - 1 || last) {
        block_barrier();
        __builtin_amdgcn_sched_barrier(0);
        const int filled = e + 1, r = lane & 31;
        Frag<T> ad0 = zero_frag<T>(), ad1 = ad0, aq0 = ad0, aq1 = ad0, bp = ad0, bs = ad0;
        if (hh == 0) {
          // entries past `filled` hold an earlier group's values or bits never
          // written: both operands are cut to the filled ones (0 * NaN is NaN)
          ad0 = frag_prefix<T>(load_frag(&sXst[1][r][0]), filled);
          ad1 = frag_prefix<T>(load_frag(&sXst[1][32 + r][0]), filled);
          aq0 = frag_prefix<T>(load_frag(&sXst[0][r][0]), filled);
          aq1 = frag_prefix<T>(load_frag(&sXst[0][32 + r][0]), filled);
          bp = frag_prefix<T>(load_frag(&sXst[2][kr][0]), filled);
          bs = frag_prefix<T>(load_frag(&sXst[3][kr][0]), filled);
        }
        mma32(dv0, ad0, bp);
        mma32(dv1, ad1, bp);
        mma32(dk0, aq0, bs);
        mma32(dk1, aq1, bs);
      }
    }
  };

  // the retriever list is staged through LDS in batches, each streamed through
  // the ring (one item in flight ahead of the compute) and drained at its end.
  // The first batch: its first copy straight from the header, its first entries
  // from the header and the rest from the list, in flight with that copy and the
  // K/V fragments (round 0's barrier makes them visible)
  for (int b0 = 0; b0 < n; b0 += NE) {
    const int nb = min(NE, n - b0);
    if (b0 == 0) {
      issue(0, enc(__builtin_amdgcn_readlane(hv, 2)));
      const int e_head = __shfl(hv, (lane + 2) & 63);  // lane i: header entry i
      if (wave == 0 && lane < kHeadEntries && lane < nb) sE[lane] = enc(e_head);
      for (int i = kHeadEntries + tid; i < nb; i += kKvThreads) sE[i] = enc(list_g[i]);
    } else {
      __syncthreads();
      for (int i = tid; i < nb; i += kKvThreads) sE[i] = enc(list_g[b0 + i]);
      __syncthreads();
      issue(0, sE[0]);
    }
    for (int u = 0; u < nb; ++u) {
      wait_vmem<0>();
      block_barrier();
      if (u + 1 < nb) issue((u + 1) & 1, sE[u + 1]);
      run(u & 1, u, u + 1 == nb);
    }
  }

  // accumulators are transposed: lane holds key kr, d = 32*dt + 8*g + 4*hh + 0..3
  const float as = p.attn_scale;
  T* dkr = dk + kr * kD;
  T* dvr = dv + kr * kD;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    store4(dvr + 8 * g + 4 * hh, dv0[4 * g], dv0[4 * g + 1], dv0[4 * g + 2], dv0[4 * g + 3]);
    store4(dvr + 32 + 8 * g + 4 * hh, dv1[4 * g], dv1[4 * g + 1], dv1[4 * g + 2], dv1[4 * g + 3]);
    store4(dkr + 8 * g + 4 * hh, as * dk0[4 * g], as * dk0[4 * g + 1], as * dk0[4 * g + 2], as * dk0[4 * g + 3]);
    store4(dkr + 32 + 8 * g + 4 * hh, as * dk1[4 * g], as * dk1[4 * g + 1], as * dk1[4 * g + 2],
           as * dk1[4 * g + 3]);
  }
}

// -------------------------------------- score and landmark gradients ----

// dw[t, s] of one row: the per-head, per-wave-half partials summed over the
// group's heads as kDwClasses interleaved classes (head h in class (h - h0) mod
// kDwClasses), each class summed in head order and the classes added in class
// order, so that both kernels that form dsel round identically.
constexpr int kDwClasses = 8;
__device__ __forceinline__ float dw_class(const float* __restrict__ dwp, int64_t b, int64_t t, int s, int H, int Hr,
                                          int hr, int64_t nQ, int K, int cls) {
  const int h0 = Hr == 1 ? 0 : hr, h1 = Hr == 1 ? H : hr + 1;
  float acc = 0.f;
  for (int h = h0 + cls; h < h1; h += kDwClasses) {
    const float* d2 = dwp + (((b * H + h) * nQ + t) * K + s) * 2;
    acc += d2[0] + d2[1];
  }
  return acc;
}

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
      for (int c = 0; c < kDwClasses; ++c) dw += dw_class(dwp, b, t, s, H, Hr, hr, nQ, K, c);
    }
  }
  float tot = ws * dw;
  tot = sum64(tot);
  if (s < K) dsel[row * K + s] = ws * (dw - tot);
}

// Weighted sum of gathered landmark rows by one 256-thread workgroup:
//   out[x] = scale * sum_u w_u src[row_u][x],  x < D,
// for the n (row, weight) pairs staged in sRow / sW.  A thread owns a 16-byte
// column block and a residue class of u (the groups), so every load is an
// independent 16-byte read and four are in flight; the groups' partial sums are
// added in a fixed order (deterministic).
constexpr int kMaxGatherPasses = 8;  // D <= 8192: at most 8 passes of 256 blocks (fp32)

template <typename T>
__device__ __forceinline__ float elem16(const u32x4& r, int m) {
  if constexpr (sizeof(T) == 2) return __uint_as_float((m & 1) ? (r[m >> 1] & 0xffff0000u) : (r[m >> 1] << 16));
  else return __uint_as_float(r[m]);
}

template <typename T>
__device__ __forceinline__ void gather_rows(const T* __restrict__ src, int D, const int64_t* sRow, const float* sW,
                                            int n, float (&acc)[kMaxGatherPasses][16 / sizeof(T)], int pass_cols,
                                            int groups) {
  constexpr int V = 16 / sizeof(T);
  const int tid = threadIdx.x, cb = tid % pass_cols, grp = tid / pass_cols;
  const int nb = D / V;
  auto ld = [&](int u, int b) { return *reinterpret_cast<const u32x4*>(src + sRow[u] * D + b * V); };
#pragma unroll
  for (int pass = 0; pass < kMaxGatherPasses; ++pass) {
    const int b = pass * pass_cols + cb;
    if (pass * pass_cols >= nb) break;
    if (grp < groups && b < nb) {
      int u = grp;
      for (; u + 3 * groups < n; u += 4 * groups) {
        const u32x4 f0 = ld(u, b), f1 = ld(u + groups, b), f2 = ld(u + 2 * groups, b), f3 = ld(u + 3 * groups, b);
        const float w0 = sW[u], w1 = sW[u + groups], w2 = sW[u + 2 * groups], w3 = sW[u + 3 * groups];
#pragma unroll
        for (int m = 0; m < V; ++m)
          acc[pass][m] += w0 * elem16<T>(f0, m) + w1 * elem16<T>(f1, m) + w2 * elem16<T>(f2, m) +
                          w3 * elem16<T>(f3, m);
      }
      for (; u < n; u += groups) {
        const u32x4 f0 = ld(u, b);
#pragma unroll
        for (int m = 0; m < V; ++m) acc[pass][m] += sW[u] * elem16<T>(f0, m);
      }
    }
  }
}

template <typename T>
__device__ __forceinline__ void gather_store(float* __restrict__ out, int D, float scale, float* sAcc,
                                             float (&acc)[kMaxGatherPasses][16 / sizeof(T)], int pass_cols,
                                             int groups) {
  constexpr int V = 16 / sizeof(T);
  const int tid = threadIdx.x, cb = tid % pass_cols, grp = tid / pass_cols;
  const int nb = D / V;
#pragma unroll
  for (int pass = 0; pass < kMaxGatherPasses; ++pass) {
    const int b = pass * pass_cols + cb;
    if (pass * pass_cols >= nb) break;
    __syncthreads();
    if (grp < groups && b < nb)
#pragma unroll
      for (int m = 0; m < V; ++m) sAcc[(grp * pass_cols + cb) * V + m] = acc[pass][m];
    __syncthreads();
    if (grp == 0 && b < nb) {
      float r[V];
#pragma unroll
      for (int m = 0; m < V; ++m) r[m] = sAcc[cb * V + m];
      for (int g = 1; g < groups; ++g)
#pragma unroll
        for (int m = 0; m < V; ++m) r[m] += sAcc[(g * pass_cols + cb) * V + m];
#pragma unroll
      for (int m = 0; m < V; m += 4)
        store4(out + b * V + m, scale * r[m], scale * r[m + 1], scale * r[m + 2], scale * r[m + 3]);
    }
  }
}

// column blocks per pass and retriever groups for a 256-thread workgroup
struct GatherShape {
  int pass_cols, groups;
};
inline GatherShape gather_shape(int D, int elem_bytes) {
  const int nb = D / (16 / elem_bytes);
  GatherShape g;
  g.pass_cols = nb < 256 ? nb : 256;
  g.groups = 256 / g.pass_cols;
  return g;
}

// dlmk_q[t] = score_scale * sum_s dsel[t, s] lmk_k[idx[t, s]]
// The row's dsel (as dsel_kernel computes it, the same summation order) is
// formed here and written out, so the backward needs no separate dsel launch
// when the landmark-query gradient is wanted: all 256 threads read the head
// classes of the dw partials, and the first wave forms dsel.
template <typename T>
__global__ __launch_bounds__(256) void dlmk_q_kernel(const T* __restrict__ lk, const int32_t* __restrict__ idx,
                                                     const float* __restrict__ w, const float* __restrict__ dwp,
                                                     float* __restrict__ dsel, float* __restrict__ dlq,
                                                     int64_t nQ, int64_t nKV, int D, int K, int H, int Hr,
                                                     int causal, float scale, GatherShape gs) {
  constexpr int V = 16 / sizeof(T);
  __shared__ int64_t sRow[32];
  __shared__ float sW[32];
  __shared__ int sN;
  __shared__ float sAcc[256 * 8];
  __shared__ float sCls[kDwClasses][32];
  const int64_t row = blockIdx.x;
  const int64_t bhr = row / nQ;
  const int64_t t = row % nQ;
  const int64_t b = bhr / Hr;
  const int hr = (int)(bhr % Hr);
  {
    // the dw partials of every head are read by all 256 threads at once: thread
    // (class c, slot s) sums head class c of slot s
    const int s = threadIdx.x & 31, c = threadIdx.x >> 5;
    sCls[c][s] = (s < K && t + causal < nQ) ? dw_class(dwp, b, t, s, H, Hr, hr, nQ, K, c) : 0.f;
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    const int s = threadIdx.x;
    float dw = 0.f, ws = 0.f;
    if (s < K) {
      ws = w[row * K + s];
      for (int c = 0; c < kDwClasses; ++c) dw += sCls[c][s];
    }
    const float tot = sum64(ws * dw);
    const float ds = ws * (dw - tot);
    if (s < K) dsel[row * K + s] = ds;
    const int j = s < K ? idx[row * K + s] : -1;
    const bool ok = j >= 0 && j < nKV;
    const uint64_t mask = __ballot(ok);
    if (ok) {
      const int rk = __popcll(mask & ((1ull << s) - 1));
      sRow[rk] = bhr * nKV + j;
      sW[rk] = ds;
    }
    if (s == 0) sN = __popcll(mask);
  }
  __syncthreads();
  float acc[kMaxGatherPasses][V];
  for (int q = 0; q < kMaxGatherPasses; ++q)
    for (int m = 0; m < V; ++m) acc[q][m] = 0.f;
  gather_rows<T>(lk, D, sRow, sW, sN, acc, gs.pass_cols, gs.groups);
  gather_store<T>(dlq + row * D, D, scale, sAcc, acc, gs.pass_cols, gs.groups);
}

// dlmk_k[j] = score_scale * sum over the rows (t, s) that retrieved j of dsel[t, s] lmk_q[t],
// in (t, s) order within each group of the list
template <typename T>
__global__ __launch_bounds__(256) void dlmk_k_kernel(const T* __restrict__ lq, const int* __restrict__ offs,
                                                     const int* __restrict__ sorted, const float* __restrict__ dsel,
                                                     float* __restrict__ dlk, int64_t nQ, int64_t nKV, int D, int K,
                                                     float scale, GatherShape gs) {
  constexpr int V = 16 / sizeof(T);
  constexpr int NB = 256;
  __shared__ int64_t sRow[NB];
  __shared__ float sW[NB];
  __shared__ float sAcc[256 * 8];
  const int64_t wid = blockIdx.x;  // (b, hr, j)
  const int64_t bhr = wid / nKV, j = wid % nKV;
  const int* off = offs + bhr * (nKV + 1);
  const int lo = off[j], hi = off[j + 1];
  const int* list = sorted + bhr * nQ * K;
  float acc[kMaxGatherPasses][V];
  for (int q = 0; q < kMaxGatherPasses; ++q)
    for (int m = 0; m < V; ++m) acc[q][m] = 0.f;
  for (int b0 = lo; b0 < hi; b0 += NB) {
    const int nb = min(NB, hi - b0);
    __syncthreads();
    if (threadIdx.x < nb) {
      const int e = list[b0 + threadIdx.x];  // t * K + s
      sRow[threadIdx.x] = bhr * nQ + e / K;
      sW[threadIdx.x] = dsel[(bhr * nQ) * K + e];
    }
    __syncthreads();
    gather_rows<T>(lq, D, sRow, sW, nb, acc, gs.pass_cols, gs.groups);
  }
  gather_store<T>(dlk + wid * D, D, scale, sAcc, acc, gs.pass_cols, gs.groups);
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

template <typename T>
hipError_t launch_bwd_t(const Shape& s, BwdParams& p, float* dsel, const void* lmk_q, const void* lmk_k,
                        float* dlmk_q, float* dlmk_k, hipStream_t st) {
  const int64_t BHr = (int64_t)s.B * s.Hr, BH = (int64_t)s.B * s.H;
  const int64_t nent = BHr * s.nQ * s.topk;
  BwdWs& w = p.ws;
  launch_kernel("weights_kernel", weights_kernel, dim3(blocks_for(nent, 256)), dim3(256), 0, st, p.idx, p.sel, w.w,
                BHr * s.nQ, s.topk, s.nKV);
  const unsigned zblocks = std::min(blocks_for(BHr * s.nKV, 256), 4096u);
  launch_kernel("fill_zero_kernel", fill_zero_kernel, dim3(zblocks), dim3(256), 0, st, w.counts, BHr * s.nKV);
  launch_kernel("csr_count_kernel", csr_count_kernel, dim3(blocks_for(nent, 256)), dim3(256), 0, st, p.idx, w.counts,
                BHr, s.nQ, s.topk, s.nKV, s.causal);
  launch_kernel("csr_scan_kernel", csr_scan_kernel, dim3((unsigned)BHr), dim3(1024), 0, st, w.counts, w.offs,
                w.cursor, s.nKV);
  launch_kernel("csr_fill_kernel", csr_fill_kernel, dim3(blocks_for(nent, 256)), dim3(256), 0, st, p.idx, w.cursor,
                w.unsorted, BHr, s.nQ, s.topk, s.nKV, s.causal);
  launch_kernel("csr_sort_kernel", csr_sort_kernel, dim3(blocks_for(BHr * s.nKV, 4)), dim3(256), 0, st, w.offs,
                w.unsorted, w.sorted, w.head, BHr, s.nQ, s.topk, s.nKV);
  const int64_t nq_work = BH * s.nQ, nk_work = BH * s.nKV;
  // persistent: kWgPerCu workgroups per CU, kPairs chunk streams each
  const int64_t dq_wgs =
      std::min<int64_t>(round8((int64_t)device_cus() * kWgPerCu), round8((nq_work + kPairs - 1) / kPairs));
  const bool xr = s.Sq != kS;  // LMK row per query chunk
  auto dq = [&](auto kernel) {
    launch_kernel("bwd_dq_kernel", kernel, dim3((unsigned)dq_wgs), dim3(kThreads), 0, st, p, nq_work);
  };
  if (s.topk <= kDqStageK)
    xr ? dq(bwd_dq_kernel<T, true, true>) : dq(bwd_dq_kernel<T, true, false>);
  else
    xr ? dq(bwd_dq_kernel<T, false, true>) : dq(bwd_dq_kernel<T, false, false>);
  auto kv = [&](auto kernel) {
    launch_kernel("bwd_dkdv_kernel", kernel, dim3((unsigned)round8(nk_work)), dim3(kKvThreads), 0, st, p, nk_work);
  };
  xr ? kv(bwd_dkdv_kernel<T, true>) : kv(bwd_dkdv_kernel<T, false>);
  if (dlmk_q) {
    // dsel is formed inside the landmark-query gradient kernel
    launch_kernel("dlmk_q_kernel", dlmk_q_kernel<T>, dim3((unsigned)(BHr * s.nQ)), dim3(256), 0, st, (const T*)lmk_k,
                  p.idx, w.w, w.dwp, dsel, dlmk_q, s.nQ, s.nKV, s.D, s.topk, s.H, s.Hr, s.causal, s.score_scale,
                  gather_shape(s.D, sizeof(T)));
  } else {
    launch_kernel("dsel_kernel", dsel_kernel, dim3((unsigned)(BHr * s.nQ)), dim3(64), 0, st, w.w, w.dwp, dsel,
                  s.nQ, s.H, s.Hr, s.topk, s.causal);
  }
  if (dlmk_k) {
    launch_kernel("dlmk_k_kernel", dlmk_k_kernel<T>, dim3((unsigned)(BHr * s.nKV)), dim3(256), 0, st, (const T*)lmk_q,
                  w.offs, w.sorted, dsel, dlmk_k, s.nQ, s.nKV, s.D, s.topk, s.score_scale,
                  gather_shape(s.D, sizeof(T)));
  }
  return take_launch_error();
}

}  // namespace

hipError_t launch_xattn_bwd(const Shape& s, const void* q, const void* k, const void* v, const int32_t* idx,
                            const float* sel, const float* lse, const void* dout, void* dq, void* dk, void* dv,
                            float* dsel, const void* lmk_q, const void* lmk_k, float* dlmk_q, float* dlmk_k,
                            void* ws, hipStream_t stream) {
  BwdParams p;
  p.q = q; p.k = k; p.v = v; p.idx = idx; p.sel = sel; p.lse = lse; p.dout = dout;
  p.dq = dq; p.dk = dk; p.dv = dv;
  p.ws = bwd_carve(s, ws);
  p.B = s.B; p.H = s.H; p.Hr = s.Hr; p.K = s.topk;
  p.nQ = s.nQ; p.nKV = s.nKV;
  p.causal = s.causal;
  p.attn_scale = s.attn_scale;
  p.windows = use_window_order(s.nKV, s.bf16 ? 2 : 4);
  return s.bf16 ? launch_bwd_t<__bf16>(s, p, dsel, lmk_q, lmk_k, dlmk_q, dlmk_k, stream)
                : launch_bwd_t<float>(s, p, dsel, lmk_q, lmk_k, dlmk_q, dlmk_k, stream);
}

}  // namespace gca
