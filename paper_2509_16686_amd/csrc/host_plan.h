// Host-side validation, plan selection and workspace layout for EG-MLA decode.
// Pure C++: no HIP calls, so it builds and is tested without a GPU.
#pragma once

#include <cstddef>
#include <cstdint>

#include "eg_mla.h"

namespace egmla {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }

// Token-tile granularity of every decode kernel.
constexpr int kTile = 32;

// Largest split-K work item (tokens); the MFMA kernel stages the slot and id
// of every token of its split in LDS.
constexpr int kMaxSplitTokens = 2048;
constexpr int kMaxSplitTokensDevice = kMaxSplitTokens;
// Largest split of the id-sliced kernel (it lists the kept tokens of its split in LDS).
constexpr int kMaxSliceSplitTokens = 4096;
// Id slices of the sliced kernel: one per XCD.
constexpr int kIdSlices = 8;

// MFMA kernel instantiations: (latent_dim, rope_dim) pairs with a compiled fast path.
bool mfma_shape_supported(const eg_mla_dims& d);
// MFMA shapes served by the token-split kernel (16 heads per work item)...
bool tok_kernel_shape(const eg_mla_dims& d);
// ... and by the head-split kernel (64 heads per work item); the others by the
// dimension-split kernel (16 heads per work item).
bool heads_kernel_shape(const eg_mla_dims& d);
constexpr int kHeadsPerItemWide = 64;
// Balanced schedule of the head-split kernel: at most this many token ranges
// (one work-group per range and block of 64 heads, one per compute unit of the
// device over all head blocks).
constexpr int kWideMaxGroups = 512;

struct DecodePlan {
  int path = EG_MLA_PATH_VALU;  // resolved: VALU or MFMA
  int split_tokens = 0;         // tokens per split-K work item
  int s_max = 0;                // splits per sequence (upper bound from the capacity)
  int capacity = 0;             // max_pages_per_seq * page_size
  int head_groups = 1;          // work items per (b, split) along heads
  int heads_per_group = 0;
  int slices = 1;               // partials per (b, split, head group): token-id slices of the sliced kernel
  bool balanced = false;        // head-split kernel: balanced schedule (split_tokens = list chunk)
  bool fused_absorb = false;    // d_c 128 split kernel absorbs the query itself (no id slices, d_h 128)
  // workspace layout (byte offsets)
  size_t off_q = 0;     // fp32 [B, H, d_c + d_r]  absorbed query | RoPE query
  size_t off_ml = 0;    // fp32 [rows, H, 2]   running max (log2 domain), sum
  size_t off_o = 0;     // fp32 [rows, H, d_c] unnormalised latent outputs
  size_t off_sched = 0; // balanced schedule: int64 [2] header, int2 [kWideMaxGroups] starts, int2 [B] rows
  size_t off_flags = 0; // fused absorption: uint64 [B, head_groups, s_max] stamps
  size_t bytes = 0;     // rows: B * s_max * slices, or kWideMaxGroups + B when balanced
};

eg_mla_status check_dims(const eg_mla_dims* d);

// Resolves `plan` (NULL = automatic) for a decode call.  Returns
// EG_MLA_ERR_UNSUPPORTED when a forced path is unavailable for the shape.
eg_mla_status make_decode_plan(const eg_mla_dims& d, int32_t batch, int32_t max_pages_per_seq,
                               const eg_mla_plan* plan, DecodePlan* out);

// Checks every host-visible argument of a decode call (pointers, sizes,
// workspace) against the resolved plan.
eg_mla_status validate_decode(const eg_mla_dims* d, int32_t batch, const void* q, const void* latent_cache,
                              const int32_t* token_id_cache, const void* gate_table, const void* w_uk,
                              const void* w_uv, const int32_t* seq_lens, int32_t max_pages_per_seq,
                              int64_t num_slots, const int32_t* page_table, const void* workspace,
                              size_t workspace_bytes, const void* out, const eg_mla_plan* plan, DecodePlan* p);

eg_mla_status validate_append(const eg_mla_dims* d, int32_t n_tokens, int32_t hidden, const void* x,
                              const int32_t* token_ids, const int32_t* positions, const int32_t* slots,
                              const void* w_dkv, const void* latent_cache, const int32_t* token_id_cache,
                              int64_t num_slots);

eg_mla_status validate_gate_rows(const eg_mla_dims* d, int32_t emb_dim, int32_t emb_vocab, int64_t n,
                                 const int32_t* ids, const void* emb, const void* w_ue, const void* out);

size_t prefill_workspace_bytes(const eg_mla_dims& d, int32_t seq_len);

eg_mla_status validate_prefill(const eg_mla_dims* d, int32_t seq_len, const void* q, const void* latent,
                               const int32_t* token_ids, const void* gate_table, const void* w_uk,
                               const void* w_uv, const void* workspace, size_t workspace_bytes,
                               const void* out);

// Batched (packed, variable-length) causal prefill on MFMA.
// Absorbed form (d_c 128, 16 heads): off_qf = absorbed queries, off_olat =
// latent outputs, off_ct = gated latents (fp16).  Explicit form (other
// shapes): off_qf = K^C, off_olat = V, off_ct = gated latents (bf16 hi rows,
// then lo rows).
struct PrefillVarlenLayout {
  size_t off_seq_start, off_qf, off_olat, off_ct = 0, bytes;
};
PrefillVarlenLayout prefill_varlen_layout(const eg_mla_dims& d, int32_t total_tokens);
bool prefill_varlen_absorbed(const eg_mla_dims& d);
bool prefill_varlen_shape_ok(const eg_mla_dims& d);
eg_mla_status validate_prefill_varlen(const eg_mla_dims* d, int32_t batch, int32_t total_tokens,
                                      const int32_t* cu_seqlens, const void* q, const void* latent,
                                      const int32_t* token_ids, const void* gate_table, const void* w_uk,
                                      const void* w_uv, const void* workspace, size_t workspace_bytes,
                                      const void* out);

// Decode with the paper-literal gate: workspace = one fp32 record per
// (sequence, 128-token tile, head): d_v centred value sums, the tile's max,
// sum of p, two pads.  LDS of the tile kernel for a head count; whether a
// layer takes the tile kernel (bf16, d_c = d_h = d_v = 128, d_r = 64, at most
// 160 heads) or the generic one, and the generic kernel's LDS.
size_t literal_workspace_bytes(const eg_mla_dims& d, int32_t batch, int32_t max_pages_per_seq);
size_t literal_lds_bytes(int num_heads);
bool literal_tile_shape(const eg_mla_dims& d);
size_t literal_generic_lds_bytes(const eg_mla_dims& d);
eg_mla_status validate_literal(const eg_mla_dims* d, int32_t batch, const void* q, const void* latent_cache,
                               const int32_t* token_id_cache, const void* gate_full, const void* w_uk,
                               const void* w_uv, const void* ln_w, const void* ln_b, uint32_t flags,
                               const int32_t* seq_lens, const int32_t* page_table, int32_t max_pages_per_seq,
                               int64_t num_slots, const void* workspace, size_t workspace_bytes, const void* out);

inline float softmax_scale(const eg_mla_dims& d) {
  if (d.softmax_scale > 0.f) return d.softmax_scale;
  return 1.0f / __builtin_sqrtf(static_cast<float>(d.head_dim + d.rope_dim));
}

inline int elem_bytes(const eg_mla_dims& d) { return d.dtype == EG_MLA_BF16 ? 2 : 4; }

// Compute units of the current device (queried once per device).
int device_cus();

}  // namespace egmla
