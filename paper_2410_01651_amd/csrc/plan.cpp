// Workspace plans and device facts shared by the C ABI and the launchers (host
// code only).
#include <atomic>

#include "gca_plan.hpp"

namespace gca {

int device_cus() {
  // one slot per device ordinal; 0 = not yet queried
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return 256;
  }
  if (dev < 64) {
    const int c = cached[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) {
    (void)hipGetLastError();
    n = 256;
  }
  if (dev < 64) cached[dev].store(n, std::memory_order_relaxed);
  return n;
}

// ----------------------------------------------------------- decode ----

DecodePlan decode_plan(const Shape& s) {
  // about 256 scan workgroups in all, every wave one contiguous range of at
  // least 64 keys
  constexpr int64_t kWaves = 4;
  const int64_t rows = (int64_t)s.B * s.Hr;
  int64_t wgs = 256 / rows;
  if (wgs < 1) wgs = 1;
  int64_t pw = (s.nKV + wgs * kWaves - 1) / (wgs * kWaves);
  if (pw < 64) pw = 64;
  pw = (pw + 7) & ~int64_t(7);
  DecodePlan p;
  p.pw = pw;
  p.wgs = ((s.nKV + pw - 1) / pw + kWaves - 1) / kWaves;
  p.lists = p.wgs * kWaves;  // a wave whose groups all lie past the keys leaves an empty list
  return p;
}

size_t decode_workspace(const Shape& s) {
  const size_t n = (size_t)s.B * s.Hr * decode_plan(s).lists * s.topk;
  return align256(n * sizeof(float)) + align256(n * sizeof(int));
}
float* decode_list_scores(const Shape&, void* ws) { return reinterpret_cast<float*>(ws); }
int* decode_list_chunks(const Shape& s, void* ws) {
  const size_t n = (size_t)s.B * s.Hr * decode_plan(s).lists * s.topk;
  return reinterpret_cast<int*>(reinterpret_cast<char*>(ws) + align256(n * sizeof(float)));
}

// ----------------------------------------------------- fused select ----

SelectPlan select_plan(const Shape& s) {
  SelectPlan p{};
  // landmark queries stay in registers (bf16 up to 512 columns, fp32 up to 256)
  // next to each lane's best-16 list at most
  p.split = s.causal && s.topk <= 16 && (s.bf16 ? s.D <= 512 : s.D <= 256);
  p.blocks = (s.nQ + kSelRows - 1) / kSelRows;
  p.tiles = (s.nKV + kSelTile - 1) / kSelTile;
  p.tiles_per_part = 64;  // a power of two
  if (!p.split) return p;
  // the largest row block needs every key tile
  const int64_t per_class = (p.tiles + kSelClasses - 1) / kSelClasses;
  p.parts_max = (per_class + p.tiles_per_part - 1) / p.tiles_per_part;
  if (p.parts_max < 1) p.parts_max = 1;
  p.lists = kSelClasses * p.parts_max;
  // items of one class: sum over row blocks of its parts there
  int64_t items = 0;
  for (int64_t r = 0; r < p.blocks; ++r) {
    // row block r reaches key chunks below its last row: tiles [0, nt)
    const int64_t last_row = (r + 1) * kSelRows - 1 < s.nQ - 1 ? (r + 1) * kSelRows - 1 : s.nQ - 1;
    int64_t nt = (last_row - 1) / kSelTile + 1;  // key chunks j <= last_row - 1
    if (last_row < 1) nt = 0;
    if (nt > p.tiles) nt = p.tiles;
    const int64_t c0 = nt > 0 ? (nt + kSelClasses - 1) / kSelClasses : 0;  // class 0 has the most tiles
    items += (c0 + p.tiles_per_part - 1) / p.tiles_per_part;
  }
  p.items_per_class = items;
  return p;
}

size_t fused_workspace(const Shape& s) {
  const SelectPlan p = select_plan(s);
  if (!p.split) return 0;
  const size_t n = (size_t)s.B * s.Hr * s.nQ * p.lists * s.topk;
  // the lists' scores and chunks, then one published threshold per row
  return align256(n * sizeof(float)) + align256(n * sizeof(int)) +
         align256(sizeof(uint32_t) * (size_t)s.B * s.Hr * s.nQ);
}

// --------------------------------------------------------- backward ----

namespace {
struct Carver {
  char* p;
  size_t used = 0;
  template <typename X>
  X* take(size_t count) {
    X* r = reinterpret_cast<X*>(p ? p + used : nullptr);
    used += align256(sizeof(X) * count);
    return r;
  }
};

BwdWs carve(const Shape& s, Carver& c) {
  const size_t BHr = (size_t)s.B * s.Hr, BH = (size_t)s.B * s.H;
  BwdWs w;
  w.w = c.take<float>(BHr * s.nQ * s.topk);
  w.Dbuf = c.take<float>(BH * s.nQ * s.Sq * s.topk);
  w.Lbuf = c.take<float>(BH * s.nQ * s.Sq * s.topk);
  w.dwp = c.take<float>(BH * s.nQ * s.topk * 2);
  w.counts = c.take<int>(BHr * s.nKV);
  w.cursor = c.take<int>(BHr * s.nKV);
  w.offs = c.take<int>(BHr * (s.nKV + 1));
  w.unsorted = c.take<int>(BHr * s.nQ * s.topk);
  w.sorted = c.take<int>(BHr * s.nQ * s.topk);
  w.head = c.take<int>(BHr * s.nKV * kHeadInts);
  return w;
}
}  // namespace

BwdWs bwd_carve(const Shape& s, void* base) {
  Carver c{reinterpret_cast<char*>(base)};
  return carve(s, c);
}

size_t bwd_workspace(const Shape& s) {
  Carver c{nullptr};
  carve(s, c);
  return c.used;
}

}  // namespace gca
