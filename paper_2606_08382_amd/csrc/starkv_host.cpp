// Host side of the C ABI: plan creation and validation, cache layout, workspace
// sizing and kernel launches.  No device allocation, no synchronization.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <algorithm>
#include <new>
#include <string>

#include "starkv.h"
#include "starkv_internal.h"

using namespace starkv;

namespace {

thread_local std::string g_last_error;

starkv_status fail(starkv_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
starkv_status fail(starkv_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

int64_t align256(int64_t x) { return (x + 255) / 256 * 256; }

// bits of the outlier and inlier regions of a quantized latent block
int hi_bits(int qmode) { return qmode == STARKV_Q_MIX8_4 ? 8 : 4; }
int lo_bits(int qmode) { return qmode == STARKV_Q_MIX4_3 ? 3 : 4; }

int outlier_channels(int qmode, int r) {
  if (qmode == STARKV_Q_MIX8_4) return 8 * ((r + 31) / 32);
  if (qmode == STARKV_Q_MIX4_3) return std::min(r, 8 * std::max(1, (r + 20) / 40));
  return 0;
}

int n_groups(int qmode, int r) {
  if (qmode == STARKV_Q_F16) return 0;
  const int ro = outlier_channels(qmode, r);
  return (ro + 31) / 32 + (r - ro + 31) / 32;
}

int row_bytes(int qmode, int r) {
  if (qmode == STARKV_Q_F16) return 2 * r;
  const int ro = outlier_channels(qmode, r);
  return ro * hi_bits(qmode) / 8 + (r - ro) * lo_bits(qmode) / 8;
}

constexpr int kLdsLimit = 160 * 1024;
constexpr int kMaxSplits = 256;         // context splits per sequence merged by the combine pass
constexpr int kComputeUnits = 256;
constexpr int kMaxSplitTokens = 8192;   // tokens per split (bounds the RoPE rotation recurrence)
constexpr int kMaxCtx = 64 * kMaxSplitTokens;   // longest context (524288 tokens)

}  // namespace

struct starkv_plan {
  starkv_config cfg;
  int32_t key_rank[STARKV_MAX_KV_HEADS];
  starkv_layout layout;
  int32_t width;          // sum_r + r_v
  // decode kernel shape
  int32_t ct, ntw, n_hg;
  int32_t hg_first[STARKV_MAX_KV_HEADS + 1];
  int32_t hg_frags[STARKV_MAX_KV_HEADS];
  int32_t hg_raw[STARKV_MAX_KV_HEADS];
  int32_t hg_mid[STARKV_MAX_KV_HEADS];
  KHeadInfo kh[STARKV_MAX_KV_HEADS];      // per slot (see the decode kernel shape)
  int32_t bk_row[STARKV_MAX_KV_HEADS];    // per KV head: first row in B_k
  int32_t cls[STARKV_MAX_KV_HEADS][2][5];
  // per processing position: the head's fields packed for the split kernel
  uint32_t o_raw[STARKV_MAX_KV_HEADS], o_geo[STARKV_MAX_KV_HEADS], o_fb[STARKV_MAX_KV_HEADS];
  uint32_t o_code[STARKV_MAX_KV_HEADS], o_meta[STARKV_MAX_KV_HEADS];
  int32_t lds_bytes;
  RowMap rmap;            // cache rows (contiguous or paged)
};

extern "C" {

const char* starkv_status_string(starkv_status s) {
  switch (s) {
    case STARKV_OK: return "ok";
    case STARKV_ERR_INVALID_ARG: return "invalid argument";
    case STARKV_ERR_UNSUPPORTED: return "unsupported configuration";
    case STARKV_ERR_CAPACITY: return "length beyond cache capacity";
    case STARKV_ERR_WORKSPACE: return "workspace missing or too small";
    case STARKV_ERR_ALIGNMENT: return "misaligned pointer";
    case STARKV_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* starkv_last_error(void) { return g_last_error.c_str(); }

starkv_status starkv_plan_create(const starkv_config* c, starkv_plan** out) {
  if (!out) return fail(STARKV_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!c) return fail(STARKV_ERR_INVALID_ARG, "config is NULL");
  if (c->batch < 1) return fail(STARKV_ERR_INVALID_ARG, "batch %d < 1", c->batch);
  if (c->n_kv_heads < 1 || c->n_q_heads < 1)
    return fail(STARKV_ERR_INVALID_ARG, "head counts must be positive");
  if (c->n_q_heads % c->n_kv_heads)
    return fail(STARKV_ERR_INVALID_ARG, "n_q_heads %d not a multiple of n_kv_heads %d",
                c->n_q_heads, c->n_kv_heads);
  if (c->head_dim < 2 || c->head_dim % 2) return fail(STARKV_ERR_INVALID_ARG, "head_dim must be even");
  if (c->capacity < 1) return fail(STARKV_ERR_INVALID_ARG, "capacity %d < 1", c->capacity);
  if (!c->key_rank) return fail(STARKV_ERR_INVALID_ARG, "key_rank is NULL");
  if (c->qmode < STARKV_Q_F16 || c->qmode > STARKV_Q_MIX4_3)
    return fail(STARKV_ERR_INVALID_ARG, "qmode %d", c->qmode);
  if (!(c->rope_theta > 1.0) || !std::isfinite(c->rope_theta))
    return fail(STARKV_ERR_INVALID_ARG, "rope_theta must be finite and > 1");
  if (c->d_model < 0) return fail(STARKV_ERR_INVALID_ARG, "d_model < 0");
  for (int dt : {c->q_dtype, c->x_dtype})
    if (dt != STARKV_DT_F16 && dt != STARKV_DT_BF16) return fail(STARKV_ERR_INVALID_ARG, "dtype %d", dt);
  if (c->out_dtype != STARKV_DT_F16 && c->out_dtype != STARKV_DT_BF16 && c->out_dtype != STARKV_DT_F32)
    return fail(STARKV_ERR_INVALID_ARG, "out_dtype %d", c->out_dtype);
  if (c->n_kv_heads > STARKV_MAX_KV_HEADS)
    return fail(STARKV_ERR_UNSUPPORTED, "n_kv_heads %d > %d", c->n_kv_heads, STARKV_MAX_KV_HEADS);
  if (c->n_q_heads > STARKV_MAX_Q_HEADS)
    return fail(STARKV_ERR_UNSUPPORTED, "n_q_heads %d > %d", c->n_q_heads, STARKV_MAX_Q_HEADS);
  const int G = c->n_q_heads / c->n_kv_heads;
  if (G > 16 || 16 % G) return fail(STARKV_ERR_UNSUPPORTED, "query heads per KV head %d not in {1,2,4,8,16}", G);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(STARKV_ERR_UNSUPPORTED, "head_dim %d not 64 or 128", c->head_dim);
  if (c->group_size != 32) return fail(STARKV_ERR_UNSUPPORTED, "group_size %d != 32", c->group_size);
  if (c->capacity > (1 << 24)) return fail(STARKV_ERR_UNSUPPORTED, "capacity %d > 2^24", c->capacity);
  const int D = c->head_dim;
  int sum_r = 0;
  for (int g = 0; g < c->n_kv_heads; ++g) {
    const int r = c->key_rank[g];
    if (r < 16 || r > D || r % 16)
      return fail(STARKV_ERR_INVALID_ARG, "key_rank[%d] = %d: need a multiple of 16 in [16, %d]", g, r, D);
    sum_r += r;
  }
  const int rv = c->value_rank;
  if (rv < 16 || rv % 16 || rv > c->n_kv_heads * D)
    return fail(STARKV_ERR_INVALID_ARG, "value_rank %d: need a multiple of 16 in [16, %d]", rv,
                c->n_kv_heads * D);
  if (rv > 1024) return fail(STARKV_ERR_UNSUPPORTED, "value_rank %d > 1024", rv);
  if (n_groups(c->qmode, rv) > 24) return fail(STARKV_ERR_UNSUPPORTED, "value_rank %d: too many groups", rv);
  if (c->page_tokens != 0) {
    const int P = c->page_tokens;
    if (P < 128 || P > 8192 || (P & (P - 1)))
      return fail(STARKV_ERR_INVALID_ARG, "page_tokens %d: need a power of two in [128, 8192]", P);
    if (c->n_pages < 1) return fail(STARKV_ERR_INVALID_ARG, "n_pages %d < 1", c->n_pages);
    if ((int64_t)c->n_pages * P > ((int64_t)1 << 31) - 1)
      return fail(STARKV_ERR_UNSUPPORTED, "page pool of %d x %d rows too large", c->n_pages, P);
    if (!c->block_table) return fail(STARKV_ERR_INVALID_ARG, "block_table is NULL");
    if (reinterpret_cast<uintptr_t>(c->block_table) % 4)
      return fail(STARKV_ERR_ALIGNMENT, "block_table not 4-byte aligned");
  }
  if (c->d_model > 0) {
    if (c->x_dtype != STARKV_DT_BF16) return fail(STARKV_ERR_UNSUPPORTED, "hidden states must be bf16");
    if (c->d_model % 8) return fail(STARKV_ERR_UNSUPPORTED, "d_model %d not a multiple of 8", c->d_model);
  }

  starkv_plan* P = new (std::nothrow) starkv_plan();
  if (!P) return fail(STARKV_ERR_INVALID_ARG, "out of host memory");
  P->cfg = *c;
  for (int g = 0; g < c->n_kv_heads; ++g) P->key_rank[g] = c->key_rank[g];
  P->cfg.key_rank = P->key_rank;
  P->width = sum_r + rv;

  // ---- layout
  starkv_layout& L = P->layout;
  std::memset(&L, 0, sizeof(L));
  const int64_t Cp = ((int64_t)c->capacity + 255) / 256 * 256;
  const bool paged = c->page_tokens != 0;
  const int64_t rows = paged ? (int64_t)c->n_pages * c->page_tokens : (int64_t)c->batch * Cp;
  L.padded_capacity = (int32_t)Cp;
  L.rows = rows;
  L.page_tokens = paged ? c->page_tokens : 0;
  L.pages_per_sequence = paged ? (c->capacity + c->page_tokens - 1) / c->page_tokens : 0;
  P->rmap.table = paged ? c->block_table : nullptr;
  P->rmap.cap_pad = (int32_t)Cp;
  P->rmap.shift = paged ? __builtin_ctz((unsigned)c->page_tokens) : 0;
  P->rmap.per_seq = L.pages_per_sequence;
  P->rmap.n_pages = paged ? c->n_pages : 0;
  L.sum_key_rank = sum_r;
  int64_t off = 0;
  for (int g = 0; g < c->n_kv_heads; ++g) {
    const int r = c->key_rank[g];
    L.key_row_bytes[g] = row_bytes(c->qmode, r);
    L.key_groups[g] = n_groups(c->qmode, r);
    L.key_outlier_channels[g] = outlier_channels(c->qmode, r);
    L.key_code_offset[g] = off;
    off = align256(off + rows * L.key_row_bytes[g]);
    L.key_meta_offset[g] = off;
    off = align256(off + rows * 4 * L.key_groups[g]);
  }
  L.value_row_bytes = row_bytes(c->qmode, rv);
  L.value_groups = n_groups(c->qmode, rv);
  L.value_outlier_channels = outlier_channels(c->qmode, rv);
  L.value_code_offset = off;
  off = align256(off + rows * L.value_row_bytes);
  L.value_meta_offset = off;
  off = align256(off + rows * 4 * L.value_groups);
  L.total_bytes = off;

  // ---- decode kernel shape: head groups whose up-projection fragments and
  // key staging fit the workgroup's LDS
  const int NT = rv / 16;
  int ntw = (NT + kWaves - 1) / kWaves;
  ntw = ntw <= 1 ? 1 : ntw <= 2 ? 2 : ntw <= 4 ? 4 : 8;
  P->ntw = ntw;
  KHeadInfo info[STARKV_MAX_KV_HEADS];   // per KV head, in head order
  int bk_row = 0;
  for (int g = 0; g < c->n_kv_heads; ++g) {
    KHeadInfo& k = info[g];
    std::memset(&k, 0, sizeof(k));
    k.code_off = L.key_code_offset[g];
    k.meta_off = L.key_meta_offset[g];
    k.head = g;
    k.rank = c->key_rank[g];
    k.nkb = (k.rank + 31) / 32;
    k.n8 = L.key_outlier_channels[g] / 8;
    k.ng8 = (L.key_outlier_channels[g] + 31) / 32;
    k.ngroups = L.key_groups[g];
    k.row_bytes = L.key_row_bytes[g];
    k.bk_row = bk_row;
    bk_row += k.rank;
  }
  // A group of KV heads [a, b) is processed by one workgroup whose waves split
  // the heads into two halves; each half owns whole score tiles (16 query
  // heads), except in a single-tile group of a kernel with at most two tiles
  // (one accumulator per half), whose second half hands its partial scores to
  // the first.  The heads are assigned to the halves to
  // balance their key work (about 2 + k-blocks units per head: the rotation is
  // per head, the reconstruction per k-block); slots list half 0's heads, then
  // half 1's.
  auto assign = [&](const int* heads, int n, int ct, int* slots, int* n_first) {
    const int tiles = (n * G + 15) / 16;
    const int cap0 = tiles < 2 ? n : std::min(n, ((tiles + 1) / 2) * 16 / G);
    int order_idx[STARKV_MAX_KV_HEADS];
    for (int i = 0; i < n; ++i) order_idx[i] = heads[i];
    std::stable_sort(order_idx, order_idx + n,
                     [&](int x, int y) { return info[x].nkb > info[y].nkb; });
    int h0[STARKV_MAX_KV_HEADS], h1[STARKV_MAX_KV_HEADS], n0 = 0, n1 = 0, w0 = 0, w1 = 0;
    for (int i = 0; i < n; ++i) {
      const int g = order_idx[i], cost = 2 + info[g].nkb;
      const bool to0 = (tiles < 2 && ct <= 2) ? w0 <= w1
                                              : n0 < cap0 && (n1 >= n - cap0 || w0 <= w1);
      if (to0) { h0[n0++] = g; w0 += cost; } else { h1[n1++] = g; w1 += cost; }
    }
    std::sort(h0, h0 + n0);
    std::sort(h1, h1 + n1);
    for (int i = 0; i < n0; ++i) slots[i] = h0[i];
    for (int i = 0; i < n1; ++i) slots[n0 + i] = h1[i];
    *n_first = n0;
  };
  auto raw_of = [&](const int* heads, int n) {
    int raw = 0;
    for (int i = 0; i < n; ++i) raw += 32 * info[heads[i]].row_bytes + 2 * info[heads[i]].ngroups * 64;
    return raw;
  };
  auto group_fits = [&](const int* heads, int n, int ct, int* frags_out, int* raw_out) {
    int frags = 0;
    for (int i = 0; i < n; ++i) frags += (D / 16) * info[heads[i]].nkb;
    int slots[STARKV_MAX_KV_HEADS], n0;
    assign(heads, n, ct, slots, &n0);
    const int raw = std::max(raw_of(slots, n0), raw_of(slots + n0, n - n0));
    *frags_out = frags;
    *raw_out = raw;
    const int nql = n * G;
    if (nql > 16 * ct) return false;
    return split_lds_bytes(frags, nql, D, ct, raw, L.value_groups, L.value_row_bytes) <= kLdsLimit;
  };
  // heads of the groups, group after group (order[first[h] ..  first[h+1]))
  int order[STARKV_MAX_KV_HEADS];
  for (int g = 0; g < c->n_kv_heads; ++g) order[g] = g;
  int best_ct = -1;
  for (int ct : {1, 2, 4}) {
    if (ct * ntw > 16) continue;
    // greedy contiguous grouping at this tile count
    int n_hg = 0, g = 0;
    bool ok = true;
    int first[STARKV_MAX_KV_HEADS + 1];
    while (g < c->n_kv_heads) {
      int e = g + 1, fr, rw;
      if (!group_fits(order + g, e - g, ct, &fr, &rw)) { ok = false; break; }
      while (e < c->n_kv_heads && group_fits(order + g, e + 1 - g, ct, &fr, &rw)) ++e;
      first[n_hg++] = g;
      g = e;
    }
    if (!ok) continue;
    first[n_hg] = c->n_kv_heads;
    if (best_ct < 0 || n_hg < P->n_hg) {
      best_ct = ct;
      P->n_hg = n_hg;
      std::memcpy(P->hg_first, first, sizeof(int) * (n_hg + 1));
    }
    if (n_hg == 1) break;
  }
  if (best_ct < 0) {
    delete P;
    return fail(STARKV_ERR_UNSUPPORTED, "no workgroup shape fits the ranks in LDS");
  }
  P->ct = best_ct;
  // All head groups run side by side for the whole split, so the split takes
  // as long as its costliest group.  With the group count fixed, the heads
  // are redistributed by cost (largest first, each into the cheapest group
  // that still fits the LDS and the tile count); the result replaces the
  // contiguous grouping when its costliest group is cheaper.
  if (P->n_hg > 1) {
    const int n_hg = P->n_hg;
    auto cost_of = [&](int g) { return 2 + info[g].nkb; };
    int worst = 0;
    for (int h = 0; h < n_hg; ++h) {
      int w = 0;
      for (int i = P->hg_first[h]; i < P->hg_first[h + 1]; ++i) w += cost_of(order[i]);
      worst = std::max(worst, w);
    }
    int by_cost[STARKV_MAX_KV_HEADS];
    for (int g = 0; g < c->n_kv_heads; ++g) by_cost[g] = g;
    std::stable_sort(by_cost, by_cost + c->n_kv_heads,
                     [&](int x, int y) { return cost_of(x) > cost_of(y); });
    int members[STARKV_MAX_KV_HEADS][STARKV_MAX_KV_HEADS], count[STARKV_MAX_KV_HEADS] = {0};
    int load[STARKV_MAX_KV_HEADS] = {0};
    bool placed_all = true;
    for (int i = 0; i < c->n_kv_heads && placed_all; ++i) {
      const int g = by_cost[i];
      int best = -1;
      for (int h = 0; h < n_hg; ++h) {
        if (best >= 0 && load[h] >= load[best]) continue;
        members[h][count[h]] = g;
        int fr, rw;
        if (group_fits(members[h], count[h] + 1, P->ct, &fr, &rw)) best = h;
      }
      if (best < 0) { placed_all = false; break; }
      members[best][count[best]++] = g;
      load[best] += cost_of(g);
    }
    int worst_lpt = 0;
    for (int h = 0; h < n_hg; ++h) worst_lpt = std::max(worst_lpt, load[h]);
    if (placed_all && worst_lpt < worst) {
      int o = 0;
      for (int h = 0; h < n_hg; ++h) {
        std::sort(members[h], members[h] + count[h]);
        P->hg_first[h] = o;
        for (int i = 0; i < count[h]; ++i) order[o++] = members[h][i];
      }
      P->hg_first[n_hg] = o;
    }
  }
  P->lds_bytes = 0;
  int pos = 0;
  for (int h = 0; h < P->n_hg; ++h) {
    const int a = P->hg_first[h], b = P->hg_first[h + 1];
    int fr, rw;
    group_fits(order + a, b - a, P->ct, &fr, &rw);
    P->hg_frags[h] = fr;
    P->hg_raw[h] = rw;
    int slots[STARKV_MAX_KV_HEADS], n0;
    assign(order + a, b - a, P->ct, slots, &n0);
    const int mid = a + n0;          // first slot of half 1
    P->hg_mid[h] = mid;
    int fb = 0;
    for (int sl = a; sl < b; ++sl) {
      KHeadInfo& k = P->kh[sl];
      k = info[slots[sl - a]];
      k.frag_base = fb;
      fb += (D / 16) * k.nkb;
    }
    for (int half = 0; half < 2; ++half) {
      const int ha = half ? mid : a, hb = half ? b : mid;
      int ro = 0;
      for (int sl = ha; sl < hb; ++sl) {
        KHeadInfo& k = P->kh[sl];
        k.raw_code = ro;
        ro += 32 * k.row_bytes;
        k.raw_meta = ro;
        ro += 2 * k.ngroups * 64;
      }
      // processing order inside the half: slots sorted by k-block count
      for (int kk = 1; kk <= 4; ++kk) {
        P->cls[h][half][kk - 1] = pos;
        for (int sl = ha; sl < hb; ++sl) {
          if (P->kh[sl].nkb != kk) continue;
          const KHeadInfo& k = P->kh[sl];
          // field widths: staging offsets < 64 KiB, row bytes < 512, rank < 256,
          // 8-bit chunks < 8, 8-bit groups < 4, groups < 8, slot < 16, planes
          // 256-byte aligned below 2^40 bytes
          const bool fits = k.raw_meta < 65536 && k.raw_code < 65536 && k.row_bytes < 512 &&
                            k.rank < 256 && k.n8 < 8 && k.ng8 < 4 && k.ngroups < 8 &&
                            sl - a < 16 && (k.code_off >> 40) == 0 && (k.meta_off >> 40) == 0 &&
                            k.code_off % 256 == 0 && k.meta_off % 256 == 0;
          if (!fits) {
            delete P;
            return fail(STARKV_ERR_UNSUPPORTED, "head parameters exceed the split kernel's table");
          }
          P->o_raw[pos] = (uint32_t)k.raw_code | ((uint32_t)k.raw_meta << 16);
          P->o_geo[pos] = (uint32_t)k.row_bytes | ((uint32_t)k.rank << 9) | ((uint32_t)k.n8 << 17) |
                          ((uint32_t)k.ng8 << 20) | ((uint32_t)k.ngroups << 22) |
                          ((uint32_t)(sl - a) << 25);
          P->o_fb[pos] = (uint32_t)k.frag_base;
          P->o_code[pos] = (uint32_t)(k.code_off >> 8);
          P->o_meta[pos] = (uint32_t)(k.meta_off >> 8);
          ++pos;
        }
      }
      P->cls[h][half][4] = pos;
    }
    const int nql = (b - a) * G;
    const int lds = split_lds_bytes(fr, nql, D, P->ct, rw, L.value_groups, L.value_row_bytes);
    if (lds > P->lds_bytes) P->lds_bytes = lds;
  }
  for (int g = 0; g < c->n_kv_heads; ++g) P->bk_row[g] = info[g].bk_row;
  *out = P;
  g_last_error.clear();
  return STARKV_OK;
}

void starkv_plan_destroy(starkv_plan* plan) { delete plan; }

size_t starkv_cache_bytes(const starkv_plan* plan) {
  return plan ? (size_t)plan->layout.total_bytes : 0;
}

starkv_status starkv_cache_layout(const starkv_plan* plan, starkv_layout* out) {
  if (!plan || !out) return fail(STARKV_ERR_INVALID_ARG, "NULL argument");
  *out = plan->layout;
  return STARKV_OK;
}

// ---------------------------------------------------------------- decode sizing

// Work plan of the split pass.  Batches of up to kMaxPlanBatch sequences use the
// device-side plan over their actual lengths: the kernels pick the split length
// S = 128 k (k >= k_lo) as the smallest giving at most `cap` work items, one
// compute unit's workgroup per item and head group (or more items where even
// 8192-token splits need them).  Larger batches split every sequence alike
// for max_ctx.
constexpr int kMaxPlanBatch = 64;
struct WorkPlan {
  bool dyn;
  int32_t k_lo, cap;
};
static WorkPlan work_plan(const starkv_plan* P, int32_t max_ctx) {
  WorkPlan w;
  const int64_t B = P->cfg.batch;
  const int64_t steps = ((int64_t)max_ctx + kStepTokens - 1) / kStepTokens;
  w.dyn = B <= kMaxPlanBatch;
  w.k_lo = (int32_t)std::max<int64_t>(1, (steps + kMaxSplits - 1) / kMaxSplits);
  const int64_t per_cu = std::max<int64_t>(1, kComputeUnits / P->n_hg);
  const int64_t at_max = B * (((int64_t)max_ctx + kMaxSplitTokens - 1) / kMaxSplitTokens);
  w.cap = (int32_t)std::max(per_cu, at_max);
  return w;
}

int32_t starkv_decode_split_tokens(const starkv_plan* P, int32_t max_ctx) {
  if (!P || max_ctx < 1) return 0;
  const WorkPlan wp = work_plan(P, max_ctx);
  if (wp.dyn) {
    // the device plan for max_ctx tokens in every sequence
    const int64_t steps = ((int64_t)max_ctx + kStepTokens - 1) / kStepTokens;
    for (int k = wp.k_lo; k < kMaxSplitTokens / kStepTokens; ++k)
      if (P->cfg.batch * ((steps + k - 1) / k) <= wp.cap) return k * kStepTokens;
    return kMaxSplitTokens;
  }
  // enough splits to give every compute unit a workgroup, at most kMaxSplits
  // per sequence (the combine pass merges up to that many)
  const int64_t wgs_per_split = (int64_t)P->cfg.batch * P->n_hg;
  int64_t splits = (kComputeUnits + wgs_per_split - 1) / wgs_per_split;
  // and enough that no split exceeds kMaxSplitTokens
  splits = std::max<int64_t>(splits, ((int64_t)max_ctx + kMaxSplitTokens - 1) / kMaxSplitTokens);
  if (splits > kMaxSplits) splits = kMaxSplits;
  int64_t len = ((int64_t)max_ctx + splits - 1) / splits;
  len = (len + kStepTokens - 1) / kStepTokens * kStepTokens;
  if (len < kStepTokens) len = kStepTokens;
  return (int32_t)len;
}

int32_t starkv_decode_splits(const starkv_plan* P, int32_t max_ctx) {
  const int32_t len = starkv_decode_split_tokens(P, max_ctx);
  if (len <= 0) return 0;
  return (max_ctx + len - 1) / len;
}

starkv_status starkv_decode_describe(const starkv_plan* P, int32_t max_ctx,
                                     starkv_decode_info* out) {
  if (!P || !out) return fail(STARKV_ERR_INVALID_ARG, "plan or out is NULL");
  if (max_ctx < 1) return fail(STARKV_ERR_INVALID_ARG, "max_ctx %d < 1", max_ctx);
  const WorkPlan wp = work_plan(P, max_ctx);
  starkv_decode_info d;
  d.head_dim = P->cfg.head_dim;
  d.qmode = P->cfg.qmode;
  d.score_tiles = P->ct;
  d.value_tiles = P->ntw;
  d.head_groups = P->n_hg;
  d.device_plan = wp.dyn ? 1 : 0;
  d.k_lo = wp.dyn ? wp.k_lo : 0;
  d.split_tokens = starkv_decode_split_tokens(P, max_ctx);
  d.items = wp.dyn ? wp.cap : P->cfg.batch * starkv_decode_splits(P, max_ctx);
  d.lds_bytes = P->lds_bytes;
  *out = d;
  return STARKV_OK;
}

// value latent, then m, l, candidate flags, unused, four candidate bounds
static int part_stride(const starkv_plan* P) { return P->cfg.value_rank + 8; }

// Work items whose partials the workspace holds: the device plan's cap, or
// every (sequence, split).
static int64_t part_slots(const starkv_plan* P, int32_t max_ctx) {
  const WorkPlan wp = work_plan(P, max_ctx);
  return wp.dyn ? wp.cap : (int64_t)P->cfg.batch * starkv_decode_splits(P, max_ctx);
}

// Workspace: the split partials [items][H_q][part_stride] fp32, then the
// rescoring candidates [items][H_q][kCand] (score, token) pairs.
static int64_t cand_offset(const starkv_plan* P, int32_t max_ctx) {
  return align256(part_slots(P, max_ctx) * P->cfg.n_q_heads * part_stride(P) * 4);
}

// Then, for the absorbed output, the normalized value latents as two fp16 parts
// [2][B][H_q * r_v].
static int64_t lat_offset(const starkv_plan* P, int32_t max_ctx) {
  return cand_offset(P, max_ctx) +
         align256(part_slots(P, max_ctx) * P->cfg.n_q_heads * kCand * 8);
}

// Then the per-sequence work plan the split pass writes for the merge pass
// [B] (first item, splits, length, 0).
static int64_t plan_offset(const starkv_plan* P, int32_t max_ctx) {
  return lat_offset(P, max_ctx) +
         align256((int64_t)2 * P->cfg.batch * P->cfg.n_q_heads * P->cfg.value_rank * 2);
}

size_t starkv_decode_workspace_bytes(const starkv_plan* P, int32_t max_ctx) {
  if (!P || max_ctx < 1) return 0;
  return (size_t)(plan_offset(P, max_ctx) + align256((int64_t)16 * P->cfg.batch));
}

static starkv_status check_common(const starkv_plan* P, int32_t max_ctx, size_t ws_bytes,
                                  const void* ws) {
  if (!P) return fail(STARKV_ERR_INVALID_ARG, "plan is NULL");
  if (max_ctx < 1) return fail(STARKV_ERR_INVALID_ARG, "max_ctx %d < 1", max_ctx);
  if (max_ctx > P->cfg.capacity)
    return fail(STARKV_ERR_CAPACITY, "max_ctx %d > capacity %d", max_ctx, P->cfg.capacity);
  if (starkv_decode_split_tokens(P, max_ctx) > kMaxSplitTokens || max_ctx > kMaxCtx)
    return fail(STARKV_ERR_UNSUPPORTED, "max_ctx %d > %d", max_ctx, kMaxCtx);
  const size_t need = starkv_decode_workspace_bytes(P, max_ctx);
  if (!ws || ws_bytes < need)
    return fail(STARKV_ERR_WORKSPACE, "decode workspace %zu bytes < %zu", ws_bytes, need);
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(STARKV_ERR_ALIGNMENT, "ws not 256-byte aligned");
  return STARKV_OK;
}

// Arguments of the decode entry points; B_v and out are checked when non-null
// is required (need_out).
static starkv_status check_decode(const starkv_plan* P, const void* cache, const void* q,
                                  const void* B_k, const void* B_v, const int32_t* ctx_len_dev,
                                  int32_t max_ctx, const void* out, const void* ws,
                                  size_t ws_bytes, bool need_out) {
  starkv_status st = check_common(P, max_ctx, ws_bytes, ws);
  if (st != STARKV_OK) return st;
  if (!cache || !q || !B_k || !ctx_len_dev || (need_out && (!B_v || !out)))
    return fail(STARKV_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(cache) % 256) return fail(STARKV_ERR_ALIGNMENT, "cache not 256-byte aligned");
  if (reinterpret_cast<uintptr_t>(q) % 16) return fail(STARKV_ERR_ALIGNMENT, "q not 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(B_k) % 16) return fail(STARKV_ERR_ALIGNMENT, "B_k not 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(ctx_len_dev) % 4) return fail(STARKV_ERR_ALIGNMENT, "ctx_len not 4-byte aligned");
  if (need_out) {
    if (reinterpret_cast<uintptr_t>(B_v) % 16) return fail(STARKV_ERR_ALIGNMENT, "B_v not 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(out) % 16) return fail(STARKV_ERR_ALIGNMENT, "out not 16-byte aligned");
  }
  return STARKV_OK;
}

static starkv_status hip_status(int e, const char* what) {
  if (e != hipSuccess) return fail(STARKV_ERR_HIP, "%s: %s", what, hipGetErrorString((hipError_t)e));
  return STARKV_OK;
}

starkv_status starkv_decode_split(const starkv_plan* P, const void* cache, const void* q,
                                  const void* B_k, const int32_t* ctx_len_dev, int32_t max_ctx,
                                  void* ws, size_t ws_bytes, starkv_stream_t stream) {
  starkv_status st = check_decode(P, cache, q, B_k, nullptr, ctx_len_dev, max_ctx, nullptr, ws,
                                  ws_bytes, false);
  if (st != STARKV_OK) return st;
  const starkv_config& c = P->cfg;
  DecodeParams p;
  std::memset(&p, 0, sizeof(p));
  p.cache = static_cast<const uint8_t*>(cache);
  p.q = q;
  p.bk = static_cast<const uint16_t*>(B_k);
  p.ctx_len = ctx_len_dev;
  p.part = static_cast<float*>(ws);
  p.cand = reinterpret_cast<float2*>(static_cast<uint8_t*>(ws) + cand_offset(P, max_ctx));
  p.plan = reinterpret_cast<int32_t*>(static_cast<uint8_t*>(ws) + plan_offset(P, max_ctx));
  p.batch = c.batch;
  p.n_q = c.n_q_heads;
  p.n_kv = c.n_kv_heads;
  p.group_q = c.n_q_heads / c.n_kv_heads;
  p.rmap = P->rmap;
  p.max_ctx = max_ctx;
  p.split_len = starkv_decode_split_tokens(P, max_ctx);
  p.n_split = starkv_decode_splits(P, max_ctx);
  {
    const WorkPlan wp = work_plan(P, max_ctx);
    p.dyn = wp.dyn;
    p.k_lo = wp.k_lo;
    p.cap = wp.cap;
  }
  p.q_bf16 = c.q_dtype == STARKV_DT_BF16;
  p.score_scale = (float)(1.4426950408889634 / std::sqrt((double)c.head_dim));
  p.log2_theta = std::log2(c.rope_theta);
  p.v_code_off = P->layout.value_code_offset;
  p.v_meta_off = P->layout.value_meta_offset;
  p.rv = c.value_rank;
  p.v_ro = P->layout.value_outlier_channels;
  p.v_ng8 = (p.v_ro + 31) / 32;
  p.v_ng = P->layout.value_groups;
  p.v_row_bytes = P->layout.value_row_bytes;
  p.part_stride = part_stride(P);
  p.n_hg = P->n_hg;
  std::memcpy(p.hg_first, P->hg_first, sizeof(p.hg_first));
  std::memcpy(p.hg_frags, P->hg_frags, sizeof(p.hg_frags));
  std::memcpy(p.hg_raw_bytes, P->hg_raw, sizeof(p.hg_raw_bytes));
  std::memcpy(p.hg_mid, P->hg_mid, sizeof(p.hg_mid));
  std::memcpy(p.kh, P->kh, sizeof(p.kh));
  std::memcpy(p.o_raw, P->o_raw, sizeof(p.o_raw));
  std::memcpy(p.o_geo, P->o_geo, sizeof(p.o_geo));
  std::memcpy(p.o_fb, P->o_fb, sizeof(p.o_fb));
  std::memcpy(p.o_code, P->o_code, sizeof(p.o_code));
  std::memcpy(p.o_meta, P->o_meta, sizeof(p.o_meta));
  std::memcpy(p.cls, P->cls, sizeof(p.cls));
  const int e = launch_decode_split_ntw(p, c.head_dim, c.qmode, P->ct, P->ntw, P->lds_bytes,
                                        static_cast<void*>(stream));
  return hip_status(e, "decode_split launch");
}

static void combine_params(const starkv_plan* P, const void* cache, const void* q,
                           const void* B_k, const void* B_v, const int32_t* ctx_len_dev,
                           int32_t max_ctx, void* out, void* ws, CombineParams& p);

starkv_status starkv_decode_combine(const starkv_plan* P, const void* cache, const void* q,
                                    const void* B_k, const void* B_v,
                                    const int32_t* ctx_len_dev, int32_t max_ctx, void* out,
                                    void* ws, size_t ws_bytes, starkv_stream_t stream) {
  starkv_status st = check_decode(P, cache, q, B_k, B_v, ctx_len_dev, max_ctx, out, ws, ws_bytes,
                                  true);
  if (st != STARKV_OK) return st;
  CombineParams p;
  combine_params(P, cache, q, B_k, B_v, ctx_len_dev, max_ctx, out, ws, p);
  return hip_status(launch_decode_combine(p, static_cast<void*>(stream)), "decode_combine launch");
}

static void combine_params(const starkv_plan* P, const void* cache, const void* q,
                           const void* B_k, const void* B_v, const int32_t* ctx_len_dev,
                           int32_t max_ctx, void* out, void* ws, CombineParams& p) {
  const starkv_config& c = P->cfg;
  const starkv_layout& L = P->layout;
  std::memset(&p, 0, sizeof(p));
  p.part = static_cast<const float*>(ws);
  p.cand = reinterpret_cast<const float2*>(static_cast<const uint8_t*>(ws) + cand_offset(P, max_ctx));
  p.plan = reinterpret_cast<const int32_t*>(static_cast<const uint8_t*>(ws) + plan_offset(P, max_ctx));
  p.bv = static_cast<const uint16_t*>(B_v);
  p.bk = static_cast<const uint16_t*>(B_k);
  p.cache = static_cast<const uint8_t*>(cache);
  p.q = q;
  p.ctx_len = ctx_len_dev;
  p.out = out;
  p.batch = c.batch;
  p.n_q = c.n_q_heads;
  p.n_kv = c.n_kv_heads;
  p.head_dim = c.head_dim;
  p.rv = c.value_rank;
  p.max_ctx = max_ctx;
  p.split_len = starkv_decode_split_tokens(P, max_ctx);
  p.n_split = starkv_decode_splits(P, max_ctx);
  {
    const WorkPlan wp = work_plan(P, max_ctx);
    p.dyn = wp.dyn;
    p.k_lo = wp.k_lo;
    p.cap = wp.cap;
    if (wp.dyn) p.n_split = kMaxSplits;   // a sequence has at most this many splits
  }
  p.part_stride = part_stride(P);
  // two workgroups per (sequence, query head), each up-projecting half of the
  // output columns, while that still leaves at least one compute unit for each
  p.col_split = 2 * (int64_t)c.batch * c.n_q_heads <= kComputeUnits ? 2 : 1;
  p.out_dtype = c.out_dtype;
  p.q_bf16 = c.q_dtype == STARKV_DT_BF16;
  p.qmode = c.qmode;
  p.rmap = P->rmap;
  p.score_scale = (float)(1.4426950408889634 / std::sqrt((double)c.head_dim));
  p.log2_theta = std::log2(c.rope_theta);
  for (int g = 0; g < c.n_kv_heads; ++g) {
    p.k_code_off[g] = L.key_code_offset[g];
    p.k_meta_off[g] = L.key_meta_offset[g];
    p.k_rank[g] = P->key_rank[g];
    p.k_ro[g] = L.key_outlier_channels[g];
    p.k_ng[g] = L.key_groups[g];
    p.k_rb[g] = L.key_row_bytes[g];
    p.k_bkrow[g] = P->bk_row[g];
    p.rmax = std::max(p.rmax, P->key_rank[g]);
  }
  p.v_code_off = L.value_code_offset;
  p.v_meta_off = L.value_meta_offset;
  p.v_ro = L.value_outlier_channels;
  p.v_ng = L.value_groups;
  p.v_rb = L.value_row_bytes;
}

starkv_status starkv_decode_attn(const starkv_plan* P, const void* cache, const void* q,
                                 const void* B_k, const void* B_v, const int32_t* ctx_len_dev,
                                 int32_t max_ctx, void* out, void* ws, size_t ws_bytes,
                                 starkv_stream_t stream) {
  starkv_status st = check_decode(P, cache, q, B_k, B_v, ctx_len_dev, max_ctx, out, ws, ws_bytes,
                                  true);
  if (st != STARKV_OK) return st;
  st = starkv_decode_split(P, cache, q, B_k, ctx_len_dev, max_ctx, ws, ws_bytes, stream);
  if (st != STARKV_OK) return st;
  return starkv_decode_combine(P, cache, q, B_k, B_v, ctx_len_dev, max_ctx, out, ws, ws_bytes,
                               stream);
}

starkv_status starkv_decode_attn_noalloc(const starkv_plan* P, const void* cache, const void* q,
                                         const void* B_k, const void* B_v,
                                         const int32_t* ctx_len_dev, int32_t max_ctx, void* out,
                                         starkv_stream_t stream) {
  if (!P) return fail(STARKV_ERR_INVALID_ARG, "plan is NULL");
  if (max_ctx < 1) return fail(STARKV_ERR_INVALID_ARG, "max_ctx %d < 1", max_ctx);
  const size_t need = starkv_decode_workspace_bytes(P, max_ctx);
  if (need > kScratchBytes)
    return fail(STARKV_ERR_WORKSPACE, "decode needs %zu workspace bytes, more than the %zu of "
                "the fixed scratch array", need, kScratchBytes);
  void* ws = nullptr;
  if (const int e = scratch_address(&ws))
    return fail(STARKV_ERR_HIP, "scratch address: %s", hipGetErrorString((hipError_t)e));
  return starkv_decode_attn(P, cache, q, B_k, B_v, ctx_len_dev, max_ctx, out, ws, kScratchBytes,
                            stream);
}

// ---------------------------------------------------------------- absorbed output

static starkv_status check_absorbed(const starkv_plan* P, const void* W_abs, int32_t d_out,
                                    const void* out) {
  if (!W_abs || !out) return fail(STARKV_ERR_INVALID_ARG, "NULL device pointer");
  if (d_out < 1) return fail(STARKV_ERR_INVALID_ARG, "d_out %d < 1", d_out);
  if ((int64_t)d_out * P->cfg.n_q_heads * P->cfg.value_rank > ((int64_t)1 << 40))
    return fail(STARKV_ERR_UNSUPPORTED, "W_abs too large");
  if (reinterpret_cast<uintptr_t>(W_abs) % 16) return fail(STARKV_ERR_ALIGNMENT, "W_abs not 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(out) % 16) return fail(STARKV_ERR_ALIGNMENT, "out not 16-byte aligned");
  return STARKV_OK;
}

starkv_status starkv_decode_combine_absorbed(const starkv_plan* P, const void* cache,
                                             const void* q, const void* B_k, const void* W_abs,
                                             int32_t d_out, const int32_t* ctx_len_dev,
                                             int32_t max_ctx, void* out, void* ws,
                                             size_t ws_bytes, starkv_stream_t stream) {
  starkv_status st = check_decode(P, cache, q, B_k, nullptr, ctx_len_dev, max_ctx, nullptr, ws,
                                  ws_bytes, false);
  if (st != STARKV_OK) return st;
  st = check_absorbed(P, W_abs, d_out, out);
  if (st != STARKV_OK) return st;
  uint16_t* lat = reinterpret_cast<uint16_t*>(static_cast<uint8_t*>(ws) + lat_offset(P, max_ctx));
  CombineParams cp;
  combine_params(P, cache, q, B_k, nullptr, ctx_len_dev, max_ctx, nullptr, ws, cp);
  cp.lat = lat;
  cp.col_split = 1;                         // one workgroup writes a head's latents
  st = hip_status(launch_decode_combine(cp, static_cast<void*>(stream)), "decode_combine launch");
  if (st != STARKV_OK) return st;
  AbsorbParams ap;
  std::memset(&ap, 0, sizeof(ap));
  ap.lat = lat;
  ap.w = static_cast<const uint16_t*>(W_abs);
  ap.out = out;
  ap.batch = P->cfg.batch;
  ap.n_out = d_out;
  ap.k = P->cfg.n_q_heads * P->cfg.value_rank;
  ap.out_dtype = P->cfg.out_dtype;
  return hip_status(launch_absorbed_out(ap, static_cast<void*>(stream)), "absorbed_out launch");
}

starkv_status starkv_decode_attn_absorbed(const starkv_plan* P, const void* cache, const void* q,
                                          const void* B_k, const void* W_abs, int32_t d_out,
                                          const int32_t* ctx_len_dev, int32_t max_ctx, void* out,
                                          void* ws, size_t ws_bytes, starkv_stream_t stream) {
  starkv_status st = check_decode(P, cache, q, B_k, nullptr, ctx_len_dev, max_ctx, nullptr, ws,
                                  ws_bytes, false);
  if (st != STARKV_OK) return st;
  st = check_absorbed(P, W_abs, d_out, out);
  if (st != STARKV_OK) return st;
  st = starkv_decode_split(P, cache, q, B_k, ctx_len_dev, max_ctx, ws, ws_bytes, stream);
  if (st != STARKV_OK) return st;
  return starkv_decode_combine_absorbed(P, cache, q, B_k, W_abs, d_out, ctx_len_dev, max_ctx, out,
                                        ws, ws_bytes, stream);
}

// ---------------------------------------------------------------- append

static void downproj_shape(const starkv_plan* P, int32_t n_new, int* k_split, int* k_chunk) {
  const int M = P->cfg.batch * n_new, N = P->width, K = P->cfg.d_model;
  if (M <= kSmallM) {            // streaming kernel: k blocks of 64 rows
    *k_chunk = 64;
    *k_split = (K + 63) / 64;
    return;
  }
  const int tiles = ((M + 63) / 64) * ((N + 63) / 64);
  int ks = 256 / tiles;
  if (ks < 1) ks = 1;
  int chunk = (K + ks - 1) / ks;
  chunk = (chunk + kDownprojK - 1) / kDownprojK * kDownprojK;
  *k_chunk = chunk;
  *k_split = (K + chunk - 1) / chunk;
}

// Appends of many tokens (a prefill) run the down-projection as one GEMM over
// all of K, with A_all transposed into the workspace.
static bool gemm_path(const starkv_plan* P, int32_t n_new) {
  return (int64_t)P->cfg.batch * n_new >= kGemmMinM && P->cfg.d_model % 64 == 0;
}

// Workspace: the fp16 latents [B*n_new][width], then either the split-k fp32
// partials or (prefill GEMM) A_all transposed, [width][d_model] bf16.
size_t starkv_append_workspace_bytes(const starkv_plan* P, int32_t n_new) {
  if (!P || n_new < 1 || P->cfg.d_model == 0) return 0;
  const int64_t mn = (int64_t)P->cfg.batch * n_new * P->width;
  if (gemm_path(P, n_new))
    return (size_t)(align256(mn * 2) + align256((int64_t)P->width * P->cfg.d_model * 2));
  int ks, kc;
  downproj_shape(P, n_new, &ks, &kc);
  return (size_t)(align256(mn * 2) + align256((int64_t)ks * mn * 4));
}

starkv_status starkv_append(const starkv_plan* P, void* cache, const void* x_or_latents,
                            const void* A_all, const int32_t* pos_dev, int32_t n_new, void* ws,
                            size_t ws_bytes, starkv_stream_t stream) {
  if (!P) return fail(STARKV_ERR_INVALID_ARG, "plan is NULL");
  if (n_new < 1) return fail(STARKV_ERR_INVALID_ARG, "n_new %d < 1", n_new);
  if (!cache || !x_or_latents || !pos_dev) return fail(STARKV_ERR_INVALID_ARG, "NULL device pointer");
  const starkv_config& c = P->cfg;
  if (c.d_model > 0 && !A_all) return fail(STARKV_ERR_INVALID_ARG, "A_all is NULL with d_model > 0");
  if (reinterpret_cast<uintptr_t>(cache) % 256) return fail(STARKV_ERR_ALIGNMENT, "cache not 256-byte aligned");
  if (reinterpret_cast<uintptr_t>(pos_dev) % 4) return fail(STARKV_ERR_ALIGNMENT, "pos not 4-byte aligned");
  const size_t need = starkv_append_workspace_bytes(P, n_new);
  if (need > 0 && (!ws || ws_bytes < need))
    return fail(STARKV_ERR_WORKSPACE, "append workspace %zu bytes < %zu", ws_bytes, need);
  if (need > 0 && reinterpret_cast<uintptr_t>(ws) % 256)
    return fail(STARKV_ERR_ALIGNMENT, "ws not 256-byte aligned");
  if ((int64_t)c.batch * n_new > (1 << 24)) return fail(STARKV_ERR_UNSUPPORTED, "too many new tokens");
  const uint16_t* lat = static_cast<const uint16_t*>(x_or_latents);
  const float* partial = nullptr;
  uint16_t* lat_out = nullptr;
  int k_split = 0;
  AppendParams a;
  std::memset(&a, 0, sizeof(a));
  a.cache = static_cast<uint8_t*>(cache);
  a.pos = pos_dev;
  a.batch = c.batch;
  a.n_new = n_new;
  a.width = P->width;
  a.capacity = c.capacity;
  a.rmap = P->rmap;
  a.qmode = c.qmode;
  a.single_writer = n_new <= 4;
  a.n_kv = c.n_kv_heads;
  {
    int lo = 0;
    a.n_items = 0;
    for (int bl = 0; bl <= c.n_kv_heads; ++bl) {
      const bool v = bl == c.n_kv_heads;
      const int r = v ? c.value_rank : c.key_rank[bl];
      a.rank[bl] = r;
      a.lat_off[bl] = lo;
      lo += r;
      a.ro[bl] = v ? P->layout.value_outlier_channels : P->layout.key_outlier_channels[bl];
      a.ng[bl] = v ? P->layout.value_groups : P->layout.key_groups[bl];
      a.row_bytes[bl] = v ? P->layout.value_row_bytes : P->layout.key_row_bytes[bl];
      a.code_off[bl] = v ? P->layout.value_code_offset : P->layout.key_code_offset[bl];
      a.meta_off[bl] = v ? P->layout.value_meta_offset : P->layout.key_meta_offset[bl];
      const int items = c.qmode == STARKV_Q_F16 ? (r + 31) / 32 : a.ng[bl];
      for (int i = 0; i < items; ++i) {
        if (a.n_items >= 128) return fail(STARKV_ERR_UNSUPPORTED, "too many quantization groups");
        a.item_block[a.n_items] = bl;
        a.item_group[a.n_items] = i;
        ++a.n_items;
      }
    }
  }
  if (c.d_model > 0) {
    if (reinterpret_cast<uintptr_t>(x_or_latents) % 16)
      return fail(STARKV_ERR_ALIGNMENT, "x not 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(A_all) % 16) return fail(STARKV_ERR_ALIGNMENT, "A_all not 16-byte aligned");
    int ks, kc;
    downproj_shape(P, n_new, &ks, &kc);
    const int64_t mn = (int64_t)c.batch * n_new * P->width;
    DownprojParams d;
    std::memset(&d, 0, sizeof(d));
    d.x = static_cast<const uint16_t*>(x_or_latents);
    d.a = static_cast<const uint16_t*>(A_all);
    d.lat = static_cast<uint16_t*>(ws);
    const bool gemm = gemm_path(P, n_new);
    if (gemm)
      d.at = reinterpret_cast<uint16_t*>(static_cast<uint8_t*>(ws) + align256(mn * 2));
    else
      d.partial = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + align256(mn * 2));
    d.m = c.batch * n_new;
    d.n = P->width;
    d.k = c.d_model;
    d.k_split = ks;
    d.k_chunk = kc;
    d.x_bf16 = 1;
    starkv_status st = hip_status(launch_downproj(d, static_cast<void*>(stream)), "downproj launch");
    if (st != STARKV_OK) return st;
    if (gemm) {                 // the latents are final: the pack reads them
      lat = d.lat;
    } else {
      lat = nullptr;
      partial = d.partial;
      lat_out = d.lat;
      k_split = ks;
    }
  } else if (reinterpret_cast<uintptr_t>(x_or_latents) % 2) {
    return fail(STARKV_ERR_ALIGNMENT, "latents not 2-byte aligned");
  }
  a.lat = lat;
  a.partial = partial;
  a.lat_out = lat_out;
  a.k_split = k_split;
  return hip_status(launch_append_pack(a, static_cast<void*>(stream)), "append pack launch");
}

starkv_status starkv_read_stream(const void* src, size_t bytes, int32_t workgroups, void* sink,
                                 size_t sink_bytes, starkv_stream_t stream) {
  if (!src || !sink) return fail(STARKV_ERR_INVALID_ARG, "NULL device pointer");
  if (bytes == 0 || bytes % 16) return fail(STARKV_ERR_INVALID_ARG, "bytes %zu: need a positive multiple of 16", bytes);
  if (workgroups == 0) workgroups = 2048;
  if (workgroups < 1 || workgroups > 65536) return fail(STARKV_ERR_INVALID_ARG, "workgroups %d", workgroups);
  if (sink_bytes < (size_t)workgroups * 16)
    return fail(STARKV_ERR_INVALID_ARG, "sink %zu bytes < %zu", sink_bytes, (size_t)workgroups * 16);
  if (reinterpret_cast<uintptr_t>(src) % 16) return fail(STARKV_ERR_ALIGNMENT, "src not 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(sink) % 4) return fail(STARKV_ERR_ALIGNMENT, "sink not 4-byte aligned");
  return hip_status(launch_read_stream(src, (int64_t)bytes, static_cast<uint32_t*>(sink), workgroups,
                                       static_cast<void*>(stream)),
                    "read_stream launch");
}

}  // extern "C"
