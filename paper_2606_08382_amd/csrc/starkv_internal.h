// Internal interface between the host library (starkv_host.cpp) and the HIP
// kernels (decode.hip, append.hip).  Not part of the public ABI.
#pragma once
#include <stdint.h>

#include "starkv.h"

namespace starkv {

constexpr int kTokenGroups = 4;          // token groups of a decode workgroup step
constexpr int kWaves = 2 * kTokenGroups;  // waves: token group x half of the KV heads
constexpr int kThreads = 64 * kWaves;
constexpr int kWaveTokens = 32;           // tokens per wave per step (two 16-token subtiles)
constexpr int kStepTokens = kTokenGroups * kWaveTokens;

// Rows of the cache planes.  Contiguous caches (table == NULL): sequence b owns
// rows b*cap_pad .. b*cap_pad + cap_pad - 1.  Paged caches: the planes have
// n_pages << shift rows, and token t of sequence b lives in row
// (table[b*per_seq + (t >> shift)] << shift) + (t & ((1 << shift) - 1)).
struct RowMap {
  const int32_t* table;
  int32_t cap_pad, shift, per_seq, n_pages;
};

#if defined(__HIP__)
// Row of token t of sequence b; page ids are clamped into the pool (the append
// kernel checks them itself and drops rows on other pages).
__device__ __forceinline__ int64_t cache_row(const RowMap& m, int b, int t) {
  if (!m.table) return (int64_t)b * m.cap_pad + t;
  int pg = m.table[(int64_t)b * m.per_seq + (t >> m.shift)];
  pg = pg < 0 ? 0 : (pg >= m.n_pages ? m.n_pages - 1 : pg);
  return ((int64_t)pg << m.shift) + (t & ((1 << m.shift) - 1));
}
#endif

// One key head as seen by the split kernel (all offsets in bytes).
struct KHeadInfo {
  int64_t code_off;      // key code plane
  int64_t meta_off;      // key meta plane
  int32_t head;          // KV head index (query heads head*G .. head*G + G - 1)
  int32_t rank;
  int32_t nkb;           // 32-channel k-blocks: ceil(rank/32)
  int32_t n8;            // 8-bit chunks (8 channels each)
  int32_t ng8;           // 8-bit groups
  int32_t ngroups;
  int32_t row_bytes;
  int32_t bk_row;        // first row of this head in B_k
  int32_t frag_base;     // first 1 KiB up-projection fragment of this head in LDS
  int32_t raw_code;      // offset of this head's codes in its wave's LDS staging area
  int32_t raw_meta;      // offset of this head's meta in its wave's LDS staging area
};

struct DecodeParams {
  const uint8_t* cache;
  const void* q;
  const uint16_t* bk;
  const int32_t* ctx_len;
  float* part;                 // split partials
  float2* cand;                // per (b, split, query head): kCand (score, token) candidates
  // work plan over ragged lengths: per sequence (first item, splits, length, 0),
  // written once (by the first wave of workgroup (0, 0)) for the merge pass
  int32_t* plan;
  int32_t batch, n_q, n_kv, group_q;   // group_q = H_q / H_kv
  RowMap rmap;
  int32_t max_ctx, split_len, n_split;
  // work plan over ragged lengths (dyn != 0, batch <= 64): grid.x = cap items,
  // the split length chosen on the device from the lengths (see the kernels);
  // otherwise grid (n_split, batch) with split_len tokens per split
  int32_t dyn, k_lo, cap;
  int32_t q_bf16;
  float score_scale;           // log2(e)/sqrt(d)
  double log2_theta;
  // values
  int64_t v_code_off, v_meta_off;
  int32_t rv, v_ro, v_ng8, v_ng, v_row_bytes;
  int32_t part_stride;         // floats per (b, split, query head)
  // head groups (blockIdx.z).  A group occupies the slots hg_first[hg] ..
  // hg_first[hg+1]-1; slot s holds KV head kh[s].head.  Each group is processed
  // in two halves (slots before and from hg_mid), each owning whole score tiles
  // of 16 query columns (slot-local query column = slot * G + j).
  int32_t n_hg;
  int32_t hg_first[STARKV_MAX_KV_HEADS + 1];
  int32_t hg_mid[STARKV_MAX_KV_HEADS];       // first slot of the second half
  int32_t hg_frags[STARKV_MAX_KV_HEADS];     // fragments used by the group
  int32_t hg_raw_bytes[STARKV_MAX_KV_HEADS]; // per-wave staging bytes (max over halves)
  KHeadInfo kh[STARKV_MAX_KV_HEADS];         // per slot
  // The heads of every half in processing order, grouped by k-block count:
  // positions cls[hg][h][k-1] .. cls[hg][h][k]-1 are the half's heads with k
  // k-blocks.  Per position, the head's fields packed for the kernel:
  //   o_raw:  staging offset of the codes | staging offset of the meta << 16
  //   o_geo:  row bytes | rank << 9 | 8-bit chunks << 17 | 8-bit groups << 20 |
  //           groups << 22 | slot within the group << 25
  //   o_fb:   first up-projection fragment
  //   o_code, o_meta: plane offsets / 256
  int32_t cls[STARKV_MAX_KV_HEADS][2][5];
  uint32_t o_raw[STARKV_MAX_KV_HEADS], o_geo[STARKV_MAX_KV_HEADS], o_fb[STARKV_MAX_KV_HEADS];
  uint32_t o_code[STARKV_MAX_KV_HEADS], o_meta[STARKV_MAX_KV_HEADS];
};

constexpr int kCand = 64;      // rescoring candidates per (sequence, split, query head):
                               // the top two scores of each of 32 lane slots
// a candidate is rescored when its share of the softmax times (1 + |score|)
// reaches this
constexpr float kRescoreTau = 1.0f / 64.0f;

struct CombineParams {
  const float* part;
  const float2* cand;
  const uint16_t* bv;
  const uint16_t* bk;
  const uint8_t* cache;
  const void* q;
  const int32_t* ctx_len;
  void* out;
  // non-NULL: write the normalized value latents a_i / l_i instead of the
  // up-projected output, as fp16 parts [2][B][H_q * r_v] (hi = fp16(x), then
  // lo = fp16(x - hi)); bv and out are unused
  uint16_t* lat;
  int32_t batch, n_q, n_kv, head_dim, rv;
  int32_t max_ctx, split_len, n_split, part_stride;
  int32_t dyn, k_lo, cap;      // as in DecodeParams
  const int32_t* plan;         // dyn: the split pass's per-sequence plan (DecodeParams::plan)
  int32_t out_dtype, q_bf16, qmode;
  int32_t rmax;                // largest key rank (sizes the rescoring buffers)
  int32_t col_split;           // workgroups per (sequence, query head), each taking
                               // head_dim / col_split output columns (1 or 2; 1 with lat)
  RowMap rmap;
  float score_scale;
  double log2_theta;
  // key head of this query head's group and the value latent (cache layout)
  int64_t k_code_off[STARKV_MAX_KV_HEADS], k_meta_off[STARKV_MAX_KV_HEADS];
  int32_t k_rank[STARKV_MAX_KV_HEADS], k_ro[STARKV_MAX_KV_HEADS], k_ng[STARKV_MAX_KV_HEADS];
  int32_t k_rb[STARKV_MAX_KV_HEADS], k_bkrow[STARKV_MAX_KV_HEADS];
  int64_t v_code_off, v_meta_off;
  int32_t v_ro, v_ng, v_rb;
};

// y [B][n_out] = lat [B][k] . w^T, w [n_out][k] fp16, lat as two fp16 parts
// (see CombineParams::lat)
struct AbsorbParams {
  const uint16_t* lat;
  const uint16_t* w;
  void* out;
  int32_t batch, n_out, k, out_dtype;
};

struct AppendParams {
  uint8_t* cache;
  const uint16_t* lat;         // fp16 latents [B][n_new][width] (when partial == NULL)
  const float* partial;        // down-projection split-k partials [k_split][B*n_new][width]
  uint16_t* lat_out;           // fp16 latents written when summing partials
  int32_t k_split;
  const int32_t* pos;
  int32_t batch, n_new, width, capacity, qmode;
  int32_t single_writer;       // every 4-bit value word has one writer (n_new <= 4)
  RowMap rmap;
  int32_t n_kv;
  // per block: 0..n_kv-1 key heads, n_kv = values
  int32_t rank[STARKV_MAX_KV_HEADS + 1];
  int32_t lat_off[STARKV_MAX_KV_HEADS + 1];
  int32_t ro[STARKV_MAX_KV_HEADS + 1];
  int32_t ng[STARKV_MAX_KV_HEADS + 1];
  int32_t row_bytes[STARKV_MAX_KV_HEADS + 1];
  int64_t code_off[STARKV_MAX_KV_HEADS + 1];
  int64_t meta_off[STARKV_MAX_KV_HEADS + 1];
  // work items per token: (block, group) pairs
  int32_t n_items;
  int32_t item_block[128];
  int32_t item_group[128];
};

struct DownprojParams {
  const uint16_t* x;           // [M][K] bf16 or fp16
  const uint16_t* a;           // [K][N] bf16
  uint16_t* at;                // non-NULL: the prefill GEMM, A transposed here ([N][K] bf16)
                               // and the latents written directly (no partials)
  float* partial;              // [ksplit][M][N]
  uint16_t* lat;               // [M][N] fp16
  int32_t m, n, k, k_split, k_chunk;
  int32_t x_bf16;
};

// launchers (return hipError_t as int)
int split_lds_bytes(int frags, int nql, int head_dim, int ct, int raw_bytes, int v_ng,
                    int v_row_bytes);
int launch_decode_split_ntw(const DecodeParams& p, int head_dim, int qmode, int ct, int ntw,
                            size_t lds_bytes, void* stream);
int launch_decode_combine(const CombineParams& p, void* stream);
// The no-allocation decode path's workspace: a fixed device array of kScratchBytes
// per device.  *out gets its device address on the current device (taken once).
constexpr size_t kScratchBytes = (size_t)32 << 20;
int scratch_address(void** out);
int launch_absorbed_out(const AbsorbParams& p, void* stream);
int launch_append_pack(const AppendParams& p, void* stream);
// rows (B * n_new) up to which the down-projection streams A_all with the
// small-M kernel: k blocks of 64 rows, one fp32 partial per block
constexpr int kSmallM = 7;
// rows from which (with d_model a multiple of 64) it is one GEMM over all of K
constexpr int kGemmMinM = 512;
// k step (and k-chunk granule) of the split-k down-projection tiles
constexpr int kDownprojK = 128;
int launch_downproj(const DownprojParams& p, void* stream);
// the plain read stream (stream.hip): bytes a multiple of 16, sink [workgroups * 4] words
int launch_read_stream(const void* src, int64_t bytes, uint32_t* sink, int workgroups,
                       void* stream);

}  // namespace starkv
