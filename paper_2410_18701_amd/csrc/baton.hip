// Host runtime of libbaton.so: handle, validation, metadata, launches.
// The C ABI is documented in include/baton.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "baton.h"
#include "common.hpp"
#include "decode_attn.hpp"
#include "decode_attn_mfma.hpp"
#include "kv_ops.hpp"
#include "layer_ops.hpp"
#include "prefill_attn.hpp"

#ifndef BATON_GQA_MFMA
#define BATON_GQA_MFMA 1   // grouped-query bf16 attention on the matrix cores
#endif
#ifndef BATON_MFMA_MIN_GROUP
#define BATON_MFMA_MIN_GROUP 2   // smallest q-heads per kv-head that takes the matrix-core kernel
#endif

#ifndef BATON_PREFILL_MFMA
#define BATON_PREFILL_MFMA 1   // bf16 prefill attention on the matrix cores (0: vector ALUs)
#endif

#ifndef BATON_PREFILL_SPLIT_LEN
#define BATON_PREFILL_SPLIT_LEN 256   // longer prompts: two key streams per prefill workgroup
#endif

static_assert(BATON_MAX_BATCH == baton::kMetaThreads, "meta kernel covers every slot");
static_assert(BATON_MAX_HOLES == baton::kMaxHoles, "hole list size");
static_assert(BATON_MAX_PREFILL == baton::kMaxPrefill, "prefill list size");

// A hole: the padding columns a prefill step inside the batch left behind the
// latest token of the rows live at that time, as absolute columns [a0, a1)
// (absolute column of logical column j: j + vend - L).
struct baton_hole {
  int64_t a0, a1, id;
};

struct baton_cache {
  baton_cache_desc d;
  int32_t esz;             // bytes per element
  int32_t vpt;             // 16-byte vectors per token row
  int32_t group;           // q-heads per kv-head
  int32_t split;           // tokens per attention work item; 0: chosen per step
  int64_t layer_vec;       // 16-byte vectors from one layer's rows of K (or V) to the next's
  int32_t step_split = 0;  // the split of the current step's work list
  int64_t L = 0;           // padded length
  int64_t base = 0;        // physical column of logical column 0
  std::vector<int32_t> lens;
  // Placeholder writes still owed by evictions: per slot, the runs [a0, a1)
  // of absolute columns its finished query's tokens occupied (its holes are
  // placeholders already).  Absolute column a lies at ring column
  // base + L - vend + a, which neither release, growth nor a step moves.
  std::vector<std::vector<std::pair<int64_t, int64_t>>> owed;
  std::vector<uint8_t> layer_done;
  int32_t n_done = 0;      // layers decoded in the current step
  // Columns appended since creation; the absolute column of logical column L.
  int64_t vend = 0;
  std::vector<baton_hole> holes;   // by id, which is also column order
  int64_t next_hole = 0;
  std::vector<int64_t> epoch;      // per slot: the holes with id >= epoch lie in its row
  // Prefill registered for the next step: prompt length per slot (0: none).
  std::vector<int32_t> plen;
  int32_t n_prefill = 0;
  int32_t step_T = 1;              // input positions per row in the next step
  // Work list of the current step as last written into a workspace.
  const void* meta_ws = nullptr;
  bool meta_valid = false;
  int32_t n_items = 0;
  int32_t n_multi = 0;     // rows with several items
  int32_t n_listed = 0;    // tokens in the gather list
  int dev = -1;            // the GPU holding K and V (found by the first no-allocation call)
};

// The work list and split-K partials of baton_decode_attn_noalloc: one array
// per GPU, held until the process ends.  Host code never passes `scratch`
// itself to a kernel (in host code it names a host-side stand-in); it uses
// the device address hipGetSymbolAddress gives for each device.
static __device__ __align__(256) uint8_t scratch[BATON_SCRATCH_BYTES];

namespace {

using baton::SegArgs;

uint32_t fill_word(const baton_cache* c) {
  if (c->esz == 4) return c->d.fill_bits;
  const uint32_t h = c->d.fill_bits & 0xFFFFu;
  return h | (h << 16);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

baton_status hip_status(hipError_t e) { return e == hipSuccess ? BATON_OK : BATON_EHIP; }

int64_t ring(int64_t x, int64_t cap) {
  x %= cap;
  return x < 0 ? x + cap : x;
}

// Index in c->holes of slot b's first hole.
int32_t first_hole(const baton_cache* c, int32_t b) {
  int32_t k = 0;
  while (k < (int32_t)c->holes.size() && c->holes[k].id < c->epoch[b]) ++k;
  return k;
}

// The holes in logical columns of the current step.
baton::HoleList hole_list(const baton_cache* c) {
  baton::HoleList hl;
  std::memset(&hl, 0, sizeof(hl));
  hl.n = (int32_t)c->holes.size();
  const int64_t shift = c->vend - c->L;
  for (int32_t k = 0; k < hl.n; ++k) {
    hl.col[k][0] = (int32_t)(c->holes[k].a0 - shift);
    hl.col[k][1] = (int32_t)(c->holes[k].a1 - shift);
  }
  return hl;
}

// Cached tokens of a live slot: its span without its holes.
int32_t row_tokens(const baton_cache* c, int32_t b, const baton::HoleList& hl) {
  const int32_t n = c->lens[b];
  if (n <= 0) return 0;
  int32_t cnt = 0;
  baton::row_runs(hl, first_hole(c, b), c->L, n, [&](int32_t t0, int32_t t1) { cnt += t1 - t0; });
  return cnt - 1;   // without the current token
}

// Forget holes that no live row holds: those released from the front, or
// older than every live row's first hole.
void drop_holes(baton_cache* c) {
  int64_t min_epoch = INT64_MAX;
  for (int32_t b = 0; b < c->d.batch; ++b)
    if (c->lens[b] > 0) min_epoch = std::min(min_epoch, c->epoch[b]);
  const int64_t shift = c->vend - c->L;
  size_t k = 0;
  while (k < c->holes.size() && (c->holes[k].id < min_epoch || c->holes[k].a1 - shift <= 0)) ++k;
  c->holes.erase(c->holes.begin(), c->holes.begin() + k);
}

#include "decode_launch.hpp"   // the decode attention's work split, workspace and launches

// Launches seg_kernel over the segments, kMaxSegs at a time.
struct Seg {
  int32_t slot, len;
  int64_t col0;
  const void* ks;   // contiguous side (null: placeholders)
  const void* vs;
  int32_t ext_len = 0;   // tokens per (layer, head) of the contiguous side; 0: len
  int32_t ext_t0 = 0;    // the segment's first token there
  int32_t dst_slot = -1; // a move: the slot receiving the columns
};

template <int VPT>
baton_status launch_segs_vpt(const baton_cache* c, const std::vector<Seg>& segs, int mode,
                             hipStream_t s) {
  constexpr int TT = baton::kCopyThreads * baton::kCopyVecs / VPT;
  for (size_t off = 0; off < segs.size(); off += baton::kMaxSegs) {
    SegArgs a;
    std::memset(&a, 0, sizeof(a));
    a.k = static_cast<uint32_t*>(c->d.k);
    a.v = static_cast<uint32_t*>(c->d.v);
    a.cap = c->d.capacity;
    a.layer_vec = c->layer_vec;
    a.n_layers = c->d.n_layers;
    a.batch = c->d.batch;
    a.n_kv_heads = c->d.n_kv_heads;
    a.fill_word = fill_word(c);
    a.extract = mode;
    const size_t n = std::min<size_t>(baton::kMaxSegs, segs.size() - off);
    int64_t tiles = 0;
    int32_t used = 0;
    for (size_t i = 0; i < n; ++i) {
      const Seg& g = segs[off + i];
      if (g.len <= 0) continue;
      const int32_t tpr = (g.len + TT - 1) / TT;
      a.slot[used] = g.slot;
      a.len[used] = g.len;
      a.col0[used] = g.col0;
      a.tiles_per_row[used] = tpr;
      a.dst_slot[used] = g.dst_slot;
      a.ext_len[used] = g.ext_len > 0 ? g.ext_len : g.len;
      a.ext_t0[used] = g.ext_t0;
      a.kext[used] = static_cast<uint32_t*>(const_cast<void*>(g.ks));
      a.vext[used] = static_cast<uint32_t*>(const_cast<void*>(g.vs));
      tiles += (int64_t)tpr * 2 * c->d.n_layers * c->d.n_kv_heads;
      a.tile_end[used] = tiles;
      ++used;
    }
    a.n_segs = used;
    if (used == 0) continue;
    if (tiles > 0x7FFFFFFF) return BATON_EINVAL;
    hipLaunchKernelGGL(baton::seg_kernel<VPT>, dim3((unsigned)tiles), dim3(baton::kCopyThreads), 0,
                       s, a);
    const baton_status st = hip_status(hipGetLastError());
    if (st != BATON_OK) return st;
  }
  return BATON_OK;
}

// mode: 0 copy into the ring (or placeholders), 1 copy out of it, 2 row to row.
baton_status launch_segs(const baton_cache* c, const std::vector<Seg>& segs, hipStream_t s,
                         int mode = 0) {
  switch (c->vpt) {
    case 8: return launch_segs_vpt<8>(c, segs, mode, s);
    case 16: return launch_segs_vpt<16>(c, segs, mode, s);
    case 32: return launch_segs_vpt<32>(c, segs, mode, s);
    default: return BATON_EDTYPE;
  }
}

template <int D, int G>
void launch_prefill_g(const baton_cache* c, baton::PrefillArgs& a, hipStream_t s) {
  const bool fa = BATON_PREFILL_MFMA && c->d.dtype == BATON_BF16;
  const int32_t per_tile = fa ? baton::kPrefillTile : baton::kWave / (D * c->esz / 16);
  int32_t tiles = 0;
  for (int32_t i = 0; i < a.n_ins; ++i) {
    tiles += (a.plen[i] + per_tile - 1) / per_tile;
    a.tile_end[i] = tiles;
  }
  const int32_t hq = c->d.n_kv_heads * G;
  a.n_tiles = tiles;
  a.n_attn = tiles * hq;
  // one XCD per kv-head's readers when the kv-heads (else the query heads) split evenly
  a.unit_heads = c->d.n_kv_heads % 8 == 0 ? G : 1;
  a.xcd_map = (hq / a.unit_heads) % 8 == 0 ? 1 : 0;
  const dim3 grid((unsigned)((int64_t)tiles * hq));
  const dim3 grid_fa((unsigned)((int64_t)tiles * (hq + c->d.n_kv_heads)));   // and the append workgroups
  int32_t longest = 0;
  for (int32_t i = 0; i < a.n_ins; ++i) longest = std::max(longest, a.plen[i]);
  if (fa && longest > BATON_PREFILL_SPLIT_LEN)
    hipLaunchKernelGGL((baton::prefill_fa_kernel<D, G, 2>), grid_fa, dim3(512), 0, s, a);
  else if (fa)
    hipLaunchKernelGGL((baton::prefill_fa_kernel<D, G, 1>), grid_fa, dim3(256), 0, s, a);
  else if (c->d.dtype == BATON_BF16)
    hipLaunchKernelGGL((baton::prefill_valu_kernel<baton::BF16Tag, D, G>), grid, dim3(baton::kWave), 0, s, a);
  else
    hipLaunchKernelGGL((baton::prefill_valu_kernel<baton::F32Tag, D, G>), grid, dim3(baton::kWave), 0, s, a);
}

template <int D>
void launch_prefill_d(const baton_cache* c, baton::PrefillArgs& a, hipStream_t s) {
  switch (c->group) {
    case 1: launch_prefill_g<D, 1>(c, a, s); break;
    case 2: launch_prefill_g<D, 2>(c, a, s); break;
    case 4: launch_prefill_g<D, 4>(c, a, s); break;
    default: launch_prefill_g<D, 8>(c, a, s); break;
  }
}

// Ring column of absolute column a.
int64_t abs_ring(const baton_cache* c, int64_t a) {
  return ring(c->base + c->L - c->vend + a, c->d.capacity);
}

// Slot b's finished query is owed placeholders: the runs of its tokens
// (its span [L - len, L) without its holes), in absolute columns.
void owe_row(baton_cache* c, int32_t b) {
  const baton::HoleList hl = hole_list(c);
  const int32_t len = c->lens[b];
  const int64_t a_row = c->vend - len;   // absolute column of the row's first token
  auto& o = c->owed[b];
  baton::row_runs(hl, first_hole(c, b), c->L, len, [&](int32_t t0, int32_t t1) {
    t1 = std::min(t1, len);   // the current column holds no token yet
    if (t1 > t0) o.push_back({a_row + t0, a_row + t1});
  });
}

// The placeholder writes slot b owes over absolute columns below `limit`
// (the rest is about to be overwritten), one segment per run.
void owed_segs(const baton_cache* c, int32_t b, int64_t limit, std::vector<Seg>& segs) {
  for (const auto& r : c->owed[b]) {
    const int64_t a1 = std::min(r.second, limit);
    if (a1 > r.first)
      segs.push_back({b, (int32_t)(a1 - r.first), abs_ring(c, r.first), nullptr, nullptr});
  }
}

// Enqueues the placeholder writes evictions still owe.
baton_status flush_pending(baton_cache* c, hipStream_t stream) {
  std::vector<Seg> segs;
  for (int32_t b = 0; b < c->d.batch; ++b) owed_segs(c, b, INT64_MAX, segs);
  if (segs.empty()) return BATON_OK;
  const baton_status st = launch_segs(c, segs, stream);
  if (st != BATON_OK) return st;
  for (auto& o : c->owed) o.clear();
  return BATON_OK;
}


// ------------------------------------------------------------ decode step --
// Argument checks shared by the decode entry points.
baton_status attn_check(const baton_cache* c, int32_t layer, const void* q, const void* k_new,
                        const void* v_new, void* out, float scale) {
  if (!c || layer < 0 || layer >= c->d.n_layers) return BATON_EINVAL;
  if (!q || !k_new || !v_new || !out) return BATON_EINVAL;
  if (!aligned16(q) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(out)) return BATON_EINVAL;
  if (!std::isfinite(scale)) return BATON_EINVAL;
  if (c->layer_done[layer]) return BATON_ESTATE;
  if (c->L + c->step_T > c->d.capacity) return BATON_ECAPACITY;
  return BATON_OK;
}

// The step's work list: meta_kernel's arguments and the counts it will produce.
void plan_items(baton_cache* c, baton::MetaArgs& m, int64_t& items, int64_t& multi, int64_t& listed) {
  std::memset(&m, 0, sizeof(m));
  m.L = c->L;
  m.batch = c->d.batch;
  c->step_split = c->split > 0 ? c->split : auto_split(c);
  m.split = c->step_split;
  m.gather_max = gather_max(c);
  m.holes = hole_list(c);
  items = multi = listed = 0;   // as meta_kernel counts them
  for (int32_t b = 0; b < c->d.batch; ++b) {
    m.lens[b] = c->plen[b] > 0 ? -1 : c->lens[b];   // a row prefilled this step has no item
    // The row's first hole, past any that ends at or before its first column:
    // meta_kernel counts every run after a row's first hole as the row's own
    // (it plans each such run once, for all the rows that hold it).
    int32_t f = first_hole(c, b);
    const int64_t c0 = m.L - std::max(m.lens[b], 0);
    while (f < m.holes.n && m.holes.col[f][1] <= c0) ++f;
    m.first[b] = (uint8_t)f;
    const baton::RowPlan p = baton::row_plan(m.holes, m.first[b], m.L, m.lens[b], m.split, m.gather_max);
    items += p.items;
    multi += p.items > 1;
    listed += p.listed;
  }
}

// The workspace laid out for exactly `items` work items and `listed` gathered tokens.
WsLayout ws_exact(const baton_cache* c, int64_t items, int64_t listed) {
  WsLayout w;
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  w.max_items = items;
  w.items_off = 0;
  w.multi_off = up(sizeof(baton::Item) * (size_t)items);
  w.gather_off = up(w.multi_off + sizeof(int4) * (size_t)c->d.batch);
  w.partial_off = up(w.gather_off + sizeof(int32_t) * (size_t)listed);
  w.total = up(w.partial_off + sizeof(float) * (size_t)c->d.n_kv_heads * items * c->group *
                                   (c->d.head_dim + 4));
  return w;
}

// One layer of the step, after the checks: the owed placeholder writes (first
// layer), the work list when `m` is given (written into the workspace at wsb
// with layout w), the attention launches, and the prefill of new queries.
baton_status attn_run(baton_cache* c, int32_t layer, const void* q, const void* k_new, const void* v_new,
                      void* out, float scale, char* wsb, const WsLayout& w, const baton::MetaArgs* m,
                      int64_t items, int64_t multi, int64_t listed, hipStream_t stream) {
  if (c->n_done == 0) {
    const baton_status st = flush_pending(c, stream);
    if (st != BATON_OK) return st;
  }
  if (m) {
    hipLaunchKernelGGL(baton::meta_kernel, dim3(1), dim3(baton::kMetaThreads), 0, stream, *m,
                       reinterpret_cast<baton::Item*>(wsb + w.items_off),
                       reinterpret_cast<int4*>(wsb + w.multi_off),
                       reinterpret_cast<int32_t*>(wsb + w.gather_off));
    const baton_status st = hip_status(hipGetLastError());
    if (st != BATON_OK) return st;
    c->n_items = (int32_t)items;
    c->n_multi = (int32_t)multi;
    c->n_listed = (int32_t)listed;
    c->meta_ws = wsb;
    c->meta_valid = true;
  }
  baton::AttnArgs a;
  std::memset(&a, 0, sizeof(a));
  // the layer's own rows
  const int64_t lw = (int64_t)layer * c->layer_vec * 4;   // 32-bit words
  a.k = static_cast<const uint32_t*>(c->d.k) + lw;
  a.k_w = static_cast<uint32_t*>(c->d.k) + lw;
  a.v = static_cast<uint32_t*>(c->d.v) + lw;
  a.q = static_cast<const uint32_t*>(q);
  a.knew = static_cast<const uint32_t*>(k_new);
  a.vnew = static_cast<const uint32_t*>(v_new);
  a.out = static_cast<uint32_t*>(out);
  a.items = reinterpret_cast<const baton::Item*>(wsb + w.items_off);
  a.multi = reinterpret_cast<const int4*>(wsb + w.multi_off);
  a.gather = reinterpret_cast<const int32_t*>(wsb + w.gather_off);
  a.partial = reinterpret_cast<float*>(wsb + w.partial_off);
  a.cap = c->d.capacity;
  a.base = c->base;
  a.L = c->L;
  a.batch = c->d.batch;
  a.n_kv_heads = c->d.n_kv_heads;
  a.split = c->step_split;
  a.n_items = c->n_items;
  a.tw = c->step_T;
  const float sc = scale == 0.f ? 1.0f / std::sqrt((float)c->d.head_dim) : scale;
  a.qscale = sc * 1.4426950408889634f;
  if (c->n_items > 0 && !launch_attn(c, a, stream)) return BATON_EDTYPE;
  baton_status st = hip_status(hipGetLastError());
  if (st != BATON_OK) return st;
  if (c->n_prefill > 0) {
    baton::PrefillArgs p;
    std::memset(&p, 0, sizeof(p));
    p.k = static_cast<uint32_t*>(c->d.k) + lw;
    p.v = static_cast<uint32_t*>(c->d.v) + lw;
    p.q = a.q;
    p.knew = a.knew;
    p.vnew = a.vnew;
    p.out = a.out;
    p.cap = c->d.capacity;
    p.base = c->base;
    p.L = c->L;
    p.T = c->step_T;
    p.batch = c->d.batch;
    p.n_kv_heads = c->d.n_kv_heads;
    p.qscale = a.qscale;
    // the prefilled queries, longest prompt first (their longest tiles are dealt first)
    for (int32_t b = 0; b < c->d.batch; ++b)
      if (c->plen[b] > 0) {
        int32_t i = p.n_ins++;
        for (; i > 0 && p.plen[i - 1] < c->plen[b]; --i) {
          p.slot[i] = p.slot[i - 1];
          p.plen[i] = p.plen[i - 1];
        }
        p.slot[i] = b;
        p.plen[i] = c->plen[b];
      }
    if (c->d.head_dim == 64) launch_prefill_d<64>(c, p, stream);
    else launch_prefill_d<128>(c, p, stream);
    st = hip_status(hipGetLastError());
    if (st != BATON_OK) return st;
  }
  c->layer_done[layer] = 1;
  ++c->n_done;
  return BATON_OK;
}

// ------------------------------------------------------ static scratch --
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];               // device address of `scratch` on each GPU
const baton_cache* g_scratch_owner[kMaxDevices]; // whose work list the scratch holds

// The scratch address on device dev, looked up once with that device current.
baton_status scratch_on(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return BATON_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return BATON_EHIP;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return BATON_EHIP;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev && hipSetDevice(cur) != hipSuccess) return BATON_EHIP;
    if (e != hipSuccess || !p) return BATON_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return BATON_OK;
}

}  // namespace

extern "C" {

const char* baton_status_string(baton_status s) {
  switch (s) {
    case BATON_OK: return "ok";
    case BATON_EINVAL: return "invalid argument";
    case BATON_ESLOT: return "slot is in the wrong state (evicting a free slot or embedding into a live one)";
    case BATON_ECAPACITY: return "padded length would exceed the ring capacity";
    case BATON_EDTYPE: return "unsupported element type, head_dim or head grouping";
    case BATON_ESTATE: return "call out of order with the decode step in progress";
    case BATON_EHIP: return "HIP runtime error";
    case BATON_ESCRATCH: return "the step's work list and partial sums exceed the static scratch";
  }
  return "unknown status";
}

baton_status baton_cache_create(const baton_cache_desc* desc, uint32_t flags, hipStream_t stream,
                                baton_cache** out) {
  if (!desc || !out) return BATON_EINVAL;
  if (flags & ~BATON_CREATE_ASSUME_FILLED) return BATON_EINVAL;
  const baton_cache_desc& d = *desc;
  if (d.dtype != BATON_F32 && d.dtype != BATON_BF16) return BATON_EDTYPE;
  if (d.head_dim != 64 && d.head_dim != 128) return BATON_EDTYPE;
  if (d.n_layers < 1 || d.batch < 1 || d.batch > BATON_MAX_BATCH || d.n_q_heads < 1 ||
      d.n_kv_heads < 1 || d.capacity < 2 || d.capacity > (int64_t(1) << 31))
    return BATON_EINVAL;
  if (d.n_q_heads % d.n_kv_heads) return BATON_EDTYPE;
  const int32_t g = d.n_q_heads / d.n_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8) return BATON_EDTYPE;
  if (!d.k || !d.v || !aligned16(d.k) || !aligned16(d.v)) return BATON_EINVAL;
  const int64_t esz = d.dtype == BATON_F32 ? 4 : 2;
  // a row of the ring is addressed with 32-bit byte offsets
  if (d.capacity * d.head_dim * esz >= (int64_t(1) << 31)) return BATON_EINVAL;
  // One layer's rows, [batch][n_kv_heads][capacity][head_dim], are dense; the
  // layers are layer_stride elements apart (0: packed), a whole number of
  // 16-byte vectors, and K's and V's layers must not overlap.
  // Sizes are bounded first so that the byte arithmetic below cannot
  // overflow: K (and V) must span less than 2^56 bytes.
  const __int128 layer_elems_w = (__int128)d.batch * d.n_kv_heads * d.capacity * d.head_dim;
  if (d.layer_stride < 0 || layer_elems_w * esz >= ((__int128)1 << 56)) return BATON_EINVAL;
  const int64_t layer_elems = (int64_t)layer_elems_w;
  const int64_t stride = d.layer_stride == 0 ? layer_elems : d.layer_stride;
  if (stride < layer_elems || (__int128)stride * esz * d.n_layers >= ((__int128)1 << 56) ||
      (stride * esz) % 16)
    return BATON_EINVAL;
  {
    const int64_t lb = layer_elems * esz, sb = stride * esz;
    const int64_t span = (int64_t)(d.n_layers - 1) * sb + lb;   // bytes from k to its last row's end
    const int64_t dist = static_cast<const char*>(d.v) - static_cast<const char*>(d.k);
    const int64_t r = ((dist % sb) + sb) % sb;             // v's offset within a layer period of k
    const bool apart = dist >= span || -dist >= span;
    const bool interleaved = d.n_layers == 1 ? (dist >= lb || -dist >= lb) : (r >= lb && r <= sb - lb);
    if (!apart && !interleaved) return BATON_EINVAL;
  }
  baton_cache* c = new (std::nothrow) baton_cache();
  if (!c) return BATON_EINVAL;
  c->d = d;
  c->esz = d.dtype == BATON_F32 ? 4 : 2;
  c->vpt = d.head_dim * c->esz / 16;
  c->layer_vec = stride * esz / 16;
  c->group = g;
  c->split = 0;
  c->lens.assign(d.batch, 0);
  c->owed.assign(d.batch, {});
  c->epoch.assign(d.batch, 0);
  c->plen.assign(d.batch, 0);
  c->layer_done.assign(d.n_layers, 0);
  if (!(flags & BATON_CREATE_ASSUME_FILLED)) {
    const int64_t n_vec = (int64_t)d.batch * d.n_kv_heads * d.capacity * c->vpt;   // per layer
    const int64_t gy = std::min<int64_t>(d.n_layers, 65535);
    const int64_t bx = std::max<int64_t>(1, std::min<int64_t>((n_vec + 255) / 256, (256 * 64 + gy - 1) / gy));
    hipLaunchKernelGGL(baton::fill_kernel, dim3((unsigned)bx, (unsigned)gy), dim3(256), 0, stream,
                       static_cast<baton::u32x4*>(d.k), static_cast<baton::u32x4*>(d.v), d.n_layers,
                       c->layer_vec, n_vec, fill_word(c));
    const baton_status st = hip_status(hipGetLastError());
    if (st != BATON_OK) {
      delete c;
      return st;
    }
  }
  *out = c;
  return BATON_OK;
}

baton_status baton_cache_destroy(baton_cache* c) {
  if (c && c->dev >= 0 && c->dev < kMaxDevices) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_owner[c->dev] == c) g_scratch_owner[c->dev] = nullptr;
  }
  delete c;
  return BATON_OK;
}

baton_status baton_kv_evict(baton_cache* c, const int32_t* slots, int32_t n, uint32_t flags,
                            hipStream_t stream) {
  if (!c || n < 0 || (n > 0 && !slots) || (flags & ~(BATON_RELEASE | BATON_SCRUB))) return BATON_EINVAL;
  if (c->n_done || c->n_prefill) return BATON_ESTATE;
  std::vector<uint8_t> seen(c->d.batch, 0);
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = slots[i];
    if (s < 0 || s >= c->d.batch || seen[s]) return BATON_EINVAL;
    seen[s] = 1;
  }
  for (int32_t i = 0; i < n; ++i)
    if (c->lens[slots[i]] == 0) return BATON_ESLOT;
  // With SCRUB the finished queries' tokens are owed placeholders (the rest of
  // their rows already holds them); the write is left to the next embed into
  // the slot, which skips the columns its own query overwrites, or to the next
  // step.  Without it they stay as they are: the mask alone excludes them.
  (void)stream;
  for (int32_t i = 0; i < n; ++i) {
    if (flags & BATON_SCRUB) owe_row(c, slots[i]);
    c->lens[slots[i]] = 0;
  }
  if (flags & BATON_RELEASE) {
    int64_t r = c->L;
    for (int32_t b = 0; b < c->d.batch; ++b)
      if (c->lens[b] > 0) r = std::min<int64_t>(r, c->L - c->lens[b]);
    c->base = ring(c->base + r, c->d.capacity);
    c->L -= r;
  }
  drop_holes(c);
  c->meta_valid = false;
  return BATON_OK;
}

baton_status baton_kv_embed(baton_cache* c, const int32_t* slots, int32_t n, const int32_t* lens,
                            const void* const* k_src, const void* const* v_src,
                            hipStream_t stream) {
  if (!c || n < 0) return BATON_EINVAL;
  if (n > 0 && (!slots || !lens || !k_src || !v_src)) return BATON_EINVAL;
  if (c->n_done || c->n_prefill) return BATON_ESTATE;
  std::vector<uint8_t> seen(c->d.batch, 0);
  int64_t longest = 0;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = slots[i];
    if (s < 0 || s >= c->d.batch || seen[s] || lens[i] < 1) return BATON_EINVAL;
    if (!k_src[i] || !v_src[i] || !aligned16(k_src[i]) || !aligned16(v_src[i])) return BATON_EINVAL;
    seen[s] = 1;
    longest = std::max<int64_t>(longest, lens[i]);
  }
  for (int32_t i = 0; i < n; ++i)
    if (c->lens[slots[i]] != 0) return BATON_ESLOT;
  const int64_t L_new = std::max(c->L, longest);
  if (L_new + 1 > c->d.capacity) return BATON_ECAPACITY;
  // Growth on the left: the new front columns come out of the unused part of
  // the ring, which holds placeholders in every row already.
  const int64_t base_new = ring(c->base - (L_new - c->L), c->d.capacity);
  // One launch: each query's copy, and the placeholders its slot still owes
  // in front of the new query (the query ends at absolute column vend, and
  // overwrites whatever is owed behind that).
  std::vector<Seg> segs;
  segs.reserve(2 * n);
  for (int32_t i = 0; i < n; ++i) {
    segs.push_back({slots[i], lens[i], ring(base_new + L_new - lens[i], c->d.capacity), k_src[i],
                    v_src[i]});
    owed_segs(c, slots[i], c->vend - lens[i], segs);
  }
  const baton_status st = launch_segs(c, segs, stream);
  if (st != BATON_OK) return st;
  c->base = base_new;
  c->L = L_new;
  for (int32_t i = 0; i < n; ++i) {
    c->lens[slots[i]] = lens[i];
    c->owed[slots[i]].clear();
    c->epoch[slots[i]] = c->next_hole;   // no earlier hole lies in its row
  }
  c->meta_valid = false;
  return BATON_OK;
}

baton_status baton_kv_extract(const baton_cache* c, const int32_t* slots, int32_t n, void* const* k_dst,
                              void* const* v_dst, hipStream_t stream) {
  if (!c || n < 0) return BATON_EINVAL;
  if (n > 0 && (!slots || !k_dst || !v_dst)) return BATON_EINVAL;
  if (c->n_done || c->n_prefill) return BATON_ESTATE;
  std::vector<uint8_t> seen(c->d.batch, 0);
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = slots[i];
    if (s < 0 || s >= c->d.batch || seen[s]) return BATON_EINVAL;
    if (!k_dst[i] || !v_dst[i] || !aligned16(k_dst[i]) || !aligned16(v_dst[i])) return BATON_EINVAL;
    seen[s] = 1;
  }
  for (int32_t i = 0; i < n; ++i)
    if (c->lens[slots[i]] == 0) return BATON_ESLOT;
  // One segment per run of consecutive tokens, packed end to end in the buffer.
  const baton::HoleList hl = hole_list(c);
  std::vector<Seg> segs;
  segs.reserve(n);
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = slots[i], len = c->lens[s];
    const int32_t ntok = row_tokens(c, s, hl);
    int32_t done = 0;
    baton::row_runs(hl, first_hole(c, s), c->L, len, [&](int32_t t0, int32_t t1) {
      t1 = std::min(t1, len);   // the current token is not cached yet
      if (t1 <= t0) return;
      Seg g{s, t1 - t0, ring(c->base + c->L - len + t0, c->d.capacity), k_dst[i], v_dst[i]};
      g.ext_len = ntok;
      g.ext_t0 = done;
      segs.push_back(g);
      done += t1 - t0;
    });
  }
  return launch_segs(c, segs, stream, /*mode=*/1);
}

baton_status baton_kv_move(baton_cache* c, const int32_t* src, const int32_t* dst, int32_t n,
                           hipStream_t stream) {
  if (!c || n < 0 || (n > 0 && (!src || !dst))) return BATON_EINVAL;
  if (c->n_done || c->n_prefill) return BATON_ESTATE;
  std::vector<uint8_t> seen(c->d.batch, 0);
  for (int32_t i = 0; i < n; ++i) {
    for (const int32_t s : {src[i], dst[i]}) {
      if (s < 0 || s >= c->d.batch || seen[s]) return BATON_EINVAL;
      seen[s] = 1;
    }
  }
  for (int32_t i = 0; i < n; ++i)
    if (c->lens[src[i]] == 0 || c->lens[dst[i]] != 0) return BATON_ESLOT;
  // The moved span ends at base + L in both rows; the columns of the target's
  // earlier query in front of it, still owed placeholders, are written in the
  // same launch.
  const int64_t end = ring(c->base + c->L, c->d.capacity);
  std::vector<Seg> copies, fills;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t len = c->lens[src[i]];
    Seg g{src[i], len, ring(end - len, c->d.capacity), nullptr, nullptr};
    g.dst_slot = dst[i];
    copies.push_back(g);
    owed_segs(c, dst[i], c->vend - len, fills);
  }
  baton_status st = launch_segs(c, copies, stream, /*mode=*/2);
  if (st == BATON_OK && !fills.empty()) st = launch_segs(c, fills, stream);
  if (st != BATON_OK) return st;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = src[i], d = dst[i];
    c->owed[d].clear();
    owe_row(c, s);   // the source's tokens are owed placeholders now
    c->lens[d] = c->lens[s];
    c->epoch[d] = c->epoch[s];
    c->lens[s] = 0;
  }
  c->meta_valid = false;
  return BATON_OK;
}

baton_status baton_shape_insert(baton_cache* c, const int32_t* slots, int32_t n, const int32_t* lens) {
  if (!c || n < 1 || n > BATON_MAX_PREFILL || !slots || !lens) return BATON_EINVAL;
  if (c->n_done) return BATON_ESTATE;
  std::vector<uint8_t> seen(c->d.batch, 0);
  int32_t T = 1;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = slots[i];
    if (s < 0 || s >= c->d.batch || seen[s] || lens[i] < 1) return BATON_EINVAL;
    seen[s] = 1;
    T = std::max(T, lens[i]);
  }
  for (int32_t i = 0; i < n; ++i)
    if (c->lens[slots[i]] != 0) return BATON_ESLOT;
  if (c->L + T > c->d.capacity) return BATON_ECAPACITY;
  // a prompt's keys of all kv-heads are addressed with 32-bit byte offsets
  if ((int64_t)T * c->d.n_kv_heads * c->d.head_dim * c->esz >= (int64_t(1) << 31)) return BATON_EINVAL;
  bool others = false;
  for (int32_t b = 0; b < c->d.batch; ++b) others |= c->lens[b] > 0;
  if (T > 1 && others && (int32_t)c->holes.size() + 1 > BATON_MAX_HOLES) return BATON_ECAPACITY;
  std::fill(c->plen.begin(), c->plen.end(), 0);
  for (int32_t i = 0; i < n; ++i) c->plen[slots[i]] = lens[i];
  c->n_prefill = n;
  c->step_T = T;
  c->meta_valid = false;
  return BATON_OK;
}

baton_status baton_build_mask(const baton_cache* c, uint8_t* mask, int64_t ld, hipStream_t stream) {
  if (!c || !mask || ld < c->L + c->step_T) return BATON_EINVAL;
  baton::MaskArgs a;
  std::memset(&a, 0, sizeof(a));
  a.mask = mask;
  a.ld = ld;
  a.L = c->L;
  a.T = c->step_T;
  a.batch = c->d.batch;
  a.holes = hole_list(c);
  for (int32_t b = 0; b < c->d.batch; ++b) {
    a.lens[b] = c->plen[b] > 0 ? -c->plen[b] : c->lens[b];
    a.first[b] = (uint8_t)first_hole(c, b);
  }
  const int64_t per_block = 256 * 4;
  const int64_t bx = std::min<int64_t>((c->L + c->step_T + per_block - 1) / per_block, 1024);
  hipLaunchKernelGGL(baton::mask_kernel, dim3((unsigned)bx, c->d.batch), dim3(256), 0, stream, a);
  return hip_status(hipGetLastError());
}

size_t baton_decode_attn_workspace_bytes(const baton_cache* c) {
  return c ? ws_layout(c).total : 0;
}

baton_status baton_decode_attn(baton_cache* c, int32_t layer, const void* q, const void* k_new,
                               const void* v_new, void* out, float scale, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  baton_status st = attn_check(c, layer, q, k_new, v_new, out, scale);
  if (st != BATON_OK) return st;
  if (!ws || !aligned16(ws)) return BATON_EINVAL;
  const WsLayout w = ws_layout(c);
  if (ws_bytes < w.total) return BATON_EINVAL;
  char* wsb = static_cast<char*>(ws);
  if (!c->meta_valid || c->meta_ws != ws) {
    baton::MetaArgs m;
    int64_t items, multi, listed;
    plan_items(c, m, items, multi, listed);
    // cannot happen: the layout bounds every row
    if (items > w.max_items || (int64_t)(w.gather_off + sizeof(int32_t) * listed) > (int64_t)w.partial_off)
      return BATON_EINVAL;
    return attn_run(c, layer, q, k_new, v_new, out, scale, wsb, w, &m, items, multi, listed, stream);
  }
  return attn_run(c, layer, q, k_new, v_new, out, scale, wsb, w, nullptr, 0, 0, 0, stream);
}

baton_status baton_decode_attn_noalloc(baton_cache* c, int32_t layer, const void* q, const void* k_new,
                                       const void* v_new, void* out, float scale, hipStream_t stream) {
  baton_status st = attn_check(c, layer, q, k_new, v_new, out, scale);
  if (st != BATON_OK) return st;
  if (c->dev < 0) {   // the GPU that holds the cache, found once
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, c->d.k) != hipSuccess) return BATON_EHIP;
    c->dev = attr.device;
  }
  void* sp = nullptr;
  st = scratch_on(c->dev, &sp);
  if (st != BATON_OK) return st;
  char* wsb = static_cast<char*>(sp);
  bool mine;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    mine = g_scratch_owner[c->dev] == c;
  }
  if (!c->meta_valid || c->meta_ws != sp || !mine) {
    // A new work list: this step's, or the scratch last held another cache's.
    baton::MetaArgs m;
    int64_t items, multi, listed;
    plan_items(c, m, items, multi, listed);
    const WsLayout w = ws_exact(c, items, listed);
    if (w.total > BATON_SCRATCH_BYTES) return BATON_ESCRATCH;
    st = attn_run(c, layer, q, k_new, v_new, out, scale, wsb, w, &m, items, multi, listed, stream);
    if (st == BATON_OK) {
      std::lock_guard<std::mutex> lock(g_scratch_mu);
      g_scratch_owner[c->dev] = c;
    }
    return st;
  }
  return attn_run(c, layer, q, k_new, v_new, out, scale, wsb, ws_exact(c, c->n_items, c->n_listed), nullptr, 0,
                  0, 0, stream);
}

baton_status baton_cache_flush(baton_cache* c, hipStream_t stream) {
  if (!c) return BATON_EINVAL;
  return flush_pending(c, stream);
}

baton_status baton_step_advance(baton_cache* c) {
  if (!c) return BATON_EINVAL;
  if (c->n_done != c->d.n_layers) return BATON_ESTATE;
  const int32_t T = c->step_T;
  if (c->n_prefill > 0) {
    // The other live rows keep padding columns L + 1 .. L + T - 1 as a hole.
    bool others = false;
    for (int32_t b = 0; b < c->d.batch; ++b) others |= c->lens[b] > 0 && c->plen[b] == 0;
    if (T > 1 && others) c->holes.push_back({c->vend + 1, c->vend + T, c->next_hole++});
    for (int32_t b = 0; b < c->d.batch; ++b) {
      if (c->plen[b] > 0) {
        c->lens[b] = c->plen[b];
        c->epoch[b] = c->next_hole;
        c->plen[b] = 0;
      } else if (c->lens[b] > 0) {
        c->lens[b] += T;
      }
    }
    c->n_prefill = 0;
    c->step_T = 1;
  } else {
    for (int32_t b = 0; b < c->d.batch; ++b)
      if (c->lens[b] > 0) c->lens[b] += 1;
  }
  c->L += T;
  c->vend += T;
  std::fill(c->layer_done.begin(), c->layer_done.end(), 0);
  c->n_done = 0;
  c->meta_valid = false;
  return BATON_OK;
}

baton_status baton_cache_query(const baton_cache* c, int64_t* L, int64_t* base, int32_t* lens) {
  if (!c) return BATON_EINVAL;
  if (L) *L = c->L;
  if (base) *base = c->base;
  if (lens) std::copy(c->lens.begin(), c->lens.end(), lens);
  return BATON_OK;
}

baton_status baton_cache_tokens(const baton_cache* c, int32_t* tokens) {
  if (!c || !tokens) return BATON_EINVAL;
  const baton::HoleList hl = hole_list(c);
  for (int32_t b = 0; b < c->d.batch; ++b) tokens[b] = row_tokens(c, b, hl);
  return BATON_OK;
}

baton_status baton_rope_qkv(const baton_cache* c, const void* qkv, void* q, void* k_new, void* v_new,
                            float theta, hipStream_t stream) {
  if (!c || !qkv || !q || !k_new || !v_new || !(theta > 1.f) || !std::isfinite(theta)) return BATON_EINVAL;
  if (c->d.dtype != BATON_BF16) return BATON_EDTYPE;
  if (c->n_prefill) return BATON_ESTATE;   // decode steps only
  baton::RopeArgs a;
  std::memset(&a, 0, sizeof(a));
  a.qkv = static_cast<const uint16_t*>(qkv);
  a.q = static_cast<uint16_t*>(q);
  a.k = static_cast<uint16_t*>(k_new);
  a.v = static_cast<uint16_t*>(v_new);
  a.n_q_heads = c->d.n_q_heads;
  a.n_kv_heads = c->d.n_kv_heads;
  a.head_dim = c->d.head_dim;
  a.log2_theta = std::log2((double)theta);
  const baton::HoleList hl = hole_list(c);
  for (int32_t b = 0; b < c->d.batch; ++b) a.pos[b] = row_tokens(c, b, hl);
  const int heads = c->d.n_q_heads + 2 * c->d.n_kv_heads;
  hipLaunchKernelGGL(baton::rope_qkv_kernel, dim3(c->d.batch * heads), dim3(baton::kWave), 0, stream, a);
  return hip_status(hipGetLastError());
}

baton_status baton_set_split_tokens(baton_cache* c, int32_t tokens) {
  if (!c || (tokens != 0 && (tokens < 64 || tokens > 4096 || tokens % 64))) return BATON_EINVAL;
  if (c->n_done) return BATON_ESTATE;
  c->split = tokens;
  c->meta_valid = false;
  return BATON_OK;
}

}  // extern "C"
