// Host side of the decode attention's launches: the automatic split of the
// work items, the workspace layout and the kernel choice by element type,
// head_dim and grouping.  Part of baton.hip's anonymous namespace (it uses the
// handle's fields); kept in a file of its own so that the kernel sources and
// this launch configuration are what the recorded HBM traffic of decode
// attention names.
#pragma once

// Automatic split: about kAutoItems work items (workgroups of
// BATON_ATTN_WAVES waves) over the step's cached tokens, which fills the GPU
// several times over at the occupancy of these kernels, never fewer than 256
// tokens per item (per-item set-up) nor more than 4096 (the tail).
#ifndef BATON_AUTO_ITEMS
#define BATON_AUTO_ITEMS 4096
#endif
#ifndef BATON_AUTO_SPLIT_MIN
#define BATON_AUTO_SPLIT_MIN 256
#endif
constexpr int64_t kAutoSplitMin = BATON_AUTO_SPLIT_MIN, kAutoSplitMax = 4096, kAutoItems = BATON_AUTO_ITEMS;

// Workspace layout: [items: max_items] [rows with several items: batch]
// [gather list: max_listed int32]
// [partials: n_kv_heads][max_items][group][head_dim + 4] fp32.
struct WsLayout {
  size_t items_off, multi_off, gather_off, partial_off, total;
  int64_t max_items;
};

int32_t gather_max(const baton_cache* c);

WsLayout ws_layout(const baton_cache* c) {
  WsLayout w;
  const int64_t B = c->d.batch;
  // Most items a row can have: its tokens cut at every split and every hole.
  const int64_t smin = c->split > 0 ? c->split : kAutoSplitMin;
  w.max_items = B * ((c->d.capacity + smin - 1) / smin + (int64_t)c->holes.size() + 1);
  // Most listed tokens: every run of every row short (below gather_max tokens).
  const int64_t max_listed = B * ((int64_t)c->holes.size() + 1) * std::max(gather_max(c) - 1, 0);
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  w.items_off = 0;
  w.multi_off = up(w.items_off + sizeof(baton::Item) * w.max_items);
  w.gather_off = up(w.multi_off + sizeof(int4) * B);
  w.partial_off = up(w.gather_off + sizeof(int32_t) * max_listed);
  w.total = up(w.partial_off + sizeof(float) * (size_t)c->d.n_kv_heads * w.max_items * c->group *
                                   (c->d.head_dim + 4));
  return w;
}

int32_t auto_split(const baton_cache* c) {
  // the tokens the step's items read: a row's span without its holes (after
  // in-batch prefill steps mostly holes), and no row prefilled in the step
  const baton::HoleList hl = hole_list(c);
  int64_t rows_tokens = 0;
  for (int32_t b = 0; b < c->d.batch; ++b)
    if (c->lens[b] > 0 && c->plen[b] == 0) rows_tokens += row_tokens(c, b, hl) + 1;
  rows_tokens *= c->d.n_kv_heads;
  int64_t s = (rows_tokens + kAutoItems - 1) / kAutoItems;
  s = (s + 63) / 64 * 64;
  return (int32_t)std::min(kAutoSplitMax, std::max(kAutoSplitMin, s));
}

// ---------------------------------------------------------------- attention --
#ifndef BATON_ATTN_U_SMALL_G
#define BATON_ATTN_U_SMALL_G 8   // token rows per lane group per iteration, G <= 2
#endif
#ifndef BATON_ATTN_U_LARGE_G
#define BATON_ATTN_U_LARGE_G 4   // G = 4, 8
#endif

#ifndef BATON_ATTN_WAVES
#define BATON_ATTN_WAVES 2       // waves per attention workgroup (one work item)
#endif

template <typename T, int D, int G>
void launch_attn_t(const baton::AttnArgs& a, int n_items, int n_multi, int hkv, hipStream_t s) {
  constexpr int U = G <= 2 ? BATON_ATTN_U_SMALL_G : BATON_ATTN_U_LARGE_G;
  constexpr int NW = BATON_ATTN_WAVES;
  const dim3 grid(n_items * hkv);
  if constexpr (BATON_GQA_MFMA && T::kBytes == 2 && G >= BATON_MFMA_MIN_GROUP)
    hipLaunchKernelGGL((baton::attn_mfma_kernel<D, G, NW>), grid, dim3(baton::kWave * NW), 0, s, a);
  else
    hipLaunchKernelGGL((baton::attn_kernel<T, D, G, U, NW>), grid, dim3(baton::kWave * NW), 0, s, a);
  if (n_multi > 0)
    hipLaunchKernelGGL((baton::combine_kernel<T, D, G>), dim3(n_multi, hkv * G), dim3(baton::kWave),
                       0, s, a);
}

template <typename T, int D>
bool launch_attn_d(int g, const baton::AttnArgs& a, int n_items, int n_multi, int hkv,
                   hipStream_t s) {
  switch (g) {
    case 1: launch_attn_t<T, D, 1>(a, n_items, n_multi, hkv, s); return true;
    case 2: launch_attn_t<T, D, 2>(a, n_items, n_multi, hkv, s); return true;
    case 4: launch_attn_t<T, D, 4>(a, n_items, n_multi, hkv, s); return true;
    case 8: launch_attn_t<T, D, 8>(a, n_items, n_multi, hkv, s); return true;
    default: return false;
  }
}

// Tokens per gathered work item: one pass of every wave of the workgroup
// (32-token blocks on the matrix-core kernel).
template <typename T, int D, int G>
constexpr int32_t gather_max_t() {
  constexpr int U = G <= 2 ? BATON_ATTN_U_SMALL_G : BATON_ATTN_U_LARGE_G;
  constexpr int32_t g = BATON_GQA_MFMA && T::kBytes == 2 && G >= BATON_MFMA_MIN_GROUP
                            ? BATON_ATTN_WAVES * 32
                            : BATON_ATTN_WAVES * baton::Geometry<T, D>::kTpi * U;
  static_assert(g <= baton::kMaxGatherTokens, "meta_kernel stages at most kMaxGatherTokens - 1 listed tokens a run");
  return g;
}

template <typename T, int D>
int32_t gather_max_d(int g) {
  switch (g) {
    case 1: return gather_max_t<T, D, 1>();
    case 2: return gather_max_t<T, D, 2>();
    case 4: return gather_max_t<T, D, 4>();
    case 8: return gather_max_t<T, D, 8>();
    default: return 0;
  }
}

int32_t gather_max(const baton_cache* c) {
  if (c->d.dtype == BATON_F32)
    return c->d.head_dim == 64 ? gather_max_d<baton::F32Tag, 64>(c->group) : gather_max_d<baton::F32Tag, 128>(c->group);
  return c->d.head_dim == 64 ? gather_max_d<baton::BF16Tag, 64>(c->group) : gather_max_d<baton::BF16Tag, 128>(c->group);
}

bool launch_attn(const baton_cache* c, const baton::AttnArgs& a, hipStream_t s) {
  const int I = c->n_items, M = c->n_multi, H = c->d.n_kv_heads;
  if (c->d.dtype == BATON_F32) {
    if (c->d.head_dim == 64) return launch_attn_d<baton::F32Tag, 64>(c->group, a, I, M, H, s);
    return launch_attn_d<baton::F32Tag, 128>(c->group, a, I, M, H, s);
  }
  if (c->d.head_dim == 64) return launch_attn_d<baton::BF16Tag, 64>(c->group, a, I, M, H, s);
  return launch_attn_d<baton::BF16Tag, 128>(c->group, a, I, M, H, s);
}

