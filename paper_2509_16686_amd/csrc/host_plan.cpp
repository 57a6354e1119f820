// Host-side validation, plan selection and workspace layout (no HIP calls).
#include "host_plan.h"

#include <algorithm>

namespace egmla {

namespace {
constexpr int kMaxRowDim = 640;     // d_c + d_r handled by the VALU kernel's LDS tile
constexpr int kMaxHeadDim = 1024;   // d_h and d_v
constexpr int kTargetWorkItems = 1024;
// Token-split MFMA kernel: one 4-wave work-group per compute unit streams
// longest without gaps between its loads (256 compute units).
constexpr int kTargetWorkItemsTok = 256;

int ceil_div(int64_t a, int64_t b) { return static_cast<int>((a + b - 1) / b); }
bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }
}  // namespace

bool mfma_shape_supported(const eg_mla_dims& d) {
  if (d.dtype != EG_MLA_BF16) return false;
  if (d.num_heads % 16 != 0) return false;
  if (d.rope_dim != 64) return false;
  return d.latent_dim == 128 || d.latent_dim == 320 || d.latent_dim == 512;
}

bool tok_kernel_shape(const eg_mla_dims& d) { return d.latent_dim == 128 && d.rope_dim == 64; }
bool heads_kernel_shape(const eg_mla_dims& d) {
  return d.latent_dim == 512 && d.rope_dim == 64 && d.head_dim == 128 && d.v_head_dim == 128 &&
         d.num_heads % kHeadsPerItemWide == 0;
}

eg_mla_status check_dims(const eg_mla_dims* d) {
  if (!d) return EG_MLA_ERR_INVALID_ARG;
  if (d->dtype != EG_MLA_FP32 && d->dtype != EG_MLA_BF16) return EG_MLA_ERR_INVALID_ARG;
  if (d->num_heads < 1 || d->head_dim < 1 || d->v_head_dim < 1 || d->latent_dim < 1 || d->rope_dim < 0 ||
      d->vocab_size < 1 || d->page_size < 1 || d->gate_dim < 1)
    return EG_MLA_ERR_INVALID_ARG;
  if (d->softmax_scale != d->softmax_scale) return EG_MLA_ERR_INVALID_ARG;  // NaN
  if (d->gate_dim != d->latent_dim) return EG_MLA_ERR_UNSUPPORTED;
  // 16-byte vector access to latent rows, gate rows and query rows.
  const int vec = d->dtype == EG_MLA_BF16 ? 8 : 4;
  if (d->latent_dim % vec != 0 || d->rope_dim % vec != 0 || d->head_dim % vec != 0)
    return EG_MLA_ERR_UNSUPPORTED;
  if (d->latent_dim + d->rope_dim > kMaxRowDim) return EG_MLA_ERR_UNSUPPORTED;
  if (d->head_dim > kMaxHeadDim || d->v_head_dim > kMaxHeadDim) return EG_MLA_ERR_UNSUPPORTED;
  return EG_MLA_OK;
}

eg_mla_status make_decode_plan(const eg_mla_dims& d, int32_t batch, int32_t max_pages_per_seq,
                               const eg_mla_plan* plan, DecodePlan* out) {
  DecodePlan p;
  const int forced = plan ? plan->path : EG_MLA_PATH_AUTO;
  if (forced != EG_MLA_PATH_AUTO && forced != EG_MLA_PATH_VALU && forced != EG_MLA_PATH_MFMA)
    return EG_MLA_ERR_INVALID_ARG;
  const bool mfma_ok = mfma_shape_supported(d);
  if (forced == EG_MLA_PATH_MFMA && !mfma_ok) return EG_MLA_ERR_UNSUPPORTED;
  p.path = (forced == EG_MLA_PATH_VALU || !mfma_ok) ? EG_MLA_PATH_VALU : EG_MLA_PATH_MFMA;

  const int64_t cap64 = static_cast<int64_t>(max_pages_per_seq) * d.page_size;
  if (cap64 > (1 << 30)) return EG_MLA_ERR_INVALID_ARG;
  p.capacity = static_cast<int>(cap64);

  if (p.path == EG_MLA_PATH_MFMA) {
    p.heads_per_group = heads_kernel_shape(d) ? kHeadsPerItemWide : 16;
  } else {
    // Heads per VALU work item: at most 8192 latent accumulators per workgroup.
    p.heads_per_group = std::max(1, std::min({d.num_heads, 8192 / d.latent_dim, 256}));
  }
  p.head_groups = ceil_div(d.num_heads, p.heads_per_group);

  const int req_slices = plan ? plan->id_slices : 0;
  if (req_slices != 0 && req_slices != 1 && req_slices != kIdSlices) return EG_MLA_ERR_INVALID_ARG;
  const bool sliced_kernel = p.path == EG_MLA_PATH_MFMA && tok_kernel_shape(d);
  // automatic: no slices (measured faster on MI355X: a sliced work item must
  // resolve its token ids before its first cache-row load)
  p.slices = sliced_kernel && req_slices == kIdSlices ? kIdSlices : 1;
  const int max_split = sliced_kernel ? kMaxSliceSplitTokens : kMaxSplitTokens;

  int split = plan ? plan->split_tokens : 0;
  if (split < 0 || split % kTile != 0) return EG_MLA_ERR_INVALID_ARG;
  if (p.path == EG_MLA_PATH_MFMA && split > max_split) return EG_MLA_ERR_UNSUPPORTED;
  if (split == 0) {
    // Work items (splits x slices) to fill the chip: each work item of the
    // sliced kernel handles 1/slices of its split's tokens.
    const int64_t work =
        static_cast<int64_t>(std::max(batch, 1)) * std::max(p.capacity, 1) * p.head_groups * p.slices;
    const int64_t target =
        p.path == EG_MLA_PATH_MFMA && (tok_kernel_shape(d) || heads_kernel_shape(d)) ? kTargetWorkItemsTok : kTargetWorkItems;
    int64_t s = (work + target - 1) / target;
    const int gran = p.slices > 1 ? 256 : kTile;  // sliced kernel: whole 256-position scan rows
    s = (s + gran - 1) / gran * gran;
    const int min_split = p.path == EG_MLA_PATH_MFMA ? 256 : 128;
    s = std::max<int64_t>(s, min_split);
    s = std::min<int64_t>(s, max_split);
    split = static_cast<int>(s);
  }
  p.split_tokens = split;
  p.s_max = std::max(1, ceil_div(std::max(p.capacity, 1), split));
  // The head-split kernel balances tokens over its work-groups whatever the
  // length mix; its split size only caps the token list it stages at a time.
  p.balanced = p.path == EG_MLA_PATH_MFMA && heads_kernel_shape(d);
  if (p.balanced && (plan == nullptr || plan->split_tokens == 0)) p.split_tokens = kMaxSplitTokens;

  const size_t B = static_cast<size_t>(std::max(batch, 0));
  const size_t H = static_cast<size_t>(d.num_heads);
  const size_t DQ = static_cast<size_t>(d.latent_dim + d.rope_dim);
  const size_t rows = p.balanced ? kWideMaxGroups + B
                                 : B * static_cast<size_t>(p.s_max) * static_cast<size_t>(p.slices);
  size_t off = 0;
  p.off_q = off;
  off = align_up(off + B * H * DQ * 4);
  p.off_ml = off;
  off = align_up(off + rows * H * 2 * 4);
  // partial outputs: fp32 sums, or (balanced schedule) fp16 rows normalised by their sums
  p.off_o = off;
  off = align_up(off + rows * H * static_cast<size_t>(d.latent_dim) * (p.balanced ? 2 : 4));
  if (p.balanced) {
    p.off_sched = off;
    off = align_up(off + 16 + kWideMaxGroups * 8 + B * 8);
  }
  // The split kernel absorbs the query itself when that costs each work-group
  // at most 2 heads' W_UK (8 to 16 splits per sequence, every split a
  // producer) and every work-group is resident at once (2 per compute unit);
  // otherwise (many splits, whose extra work-groups only wait, or a batch of
  // several rounds of work-groups each reading 4 or more heads' W_UK) the
  // absorption kernel runs first (measured: B32 L4096 25.2 against 25.7 us
  // per call; B4 L32768 28.9 against 27.8; B256 L2048 70.8 against 59.4).
  const int64_t nblk = static_cast<int64_t>(std::max(batch, 0)) * p.s_max * p.head_groups;
  p.fused_absorb = sliced_kernel && p.slices == 1 && d.head_dim == 128 && p.s_max >= 8 && p.s_max <= 16 &&
                   nblk <= 2 * kTargetWorkItemsTok;
  if (p.fused_absorb) {
    p.off_flags = off;
    off = align_up(off + B * static_cast<size_t>(p.head_groups) * static_cast<size_t>(p.s_max) * 8);
  }
  p.bytes = std::max<size_t>(off, kAlign);
  *out = p;
  return EG_MLA_OK;
}

eg_mla_status validate_decode(const eg_mla_dims* d, int32_t batch, const void* q, const void* latent_cache,
                              const int32_t* token_id_cache, const void* gate_table, const void* w_uk,
                              const void* w_uv, const int32_t* seq_lens, int32_t max_pages_per_seq,
                              int64_t num_slots, const int32_t* page_table, const void* workspace,
                              size_t workspace_bytes, const void* out, const eg_mla_plan* plan, DecodePlan* p) {
  eg_mla_status st = check_dims(d);
  if (st != EG_MLA_OK) return st;
  if (batch < 0 || max_pages_per_seq < 0 || num_slots < 0) return EG_MLA_ERR_INVALID_ARG;
  if (num_slots >= (int64_t{1} << 31)) return EG_MLA_ERR_UNSUPPORTED;  // 32-bit row indices in the kernels
  st = make_decode_plan(*d, batch, max_pages_per_seq, plan, p);
  if (st != EG_MLA_OK) return st;
  if (batch == 0) return EG_MLA_OK;
  if (!q || !gate_table || !w_uk || !w_uv || !seq_lens || !out) return EG_MLA_ERR_INVALID_ARG;
  if (max_pages_per_seq > 0 && (!latent_cache || !token_id_cache)) return EG_MLA_ERR_INVALID_ARG;
  if (!page_table) {
    // contiguous rows: every sequence's capacity must fit in the cache
    const int64_t need = static_cast<int64_t>(batch) * max_pages_per_seq * d->page_size;
    if (need > num_slots) return EG_MLA_ERR_INVALID_ARG;
  } else if (num_slots < d->page_size && max_pages_per_seq > 0) {
    return EG_MLA_ERR_INVALID_ARG;
  }
  // 16-byte vector loads of rows and weights
  if (!aligned16(q) || !aligned16(latent_cache) || !aligned16(gate_table) || !aligned16(w_uk) || !aligned16(w_uv))
    return EG_MLA_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < p->bytes) return EG_MLA_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return EG_MLA_ERR_WORKSPACE;
  return EG_MLA_OK;
}

eg_mla_status validate_append(const eg_mla_dims* d, int32_t n_tokens, int32_t hidden, const void* x,
                              const int32_t* token_ids, const int32_t* positions, const int32_t* slots,
                              const void* w_dkv, const void* latent_cache, const int32_t* token_id_cache,
                              int64_t num_slots) {
  eg_mla_status st = check_dims(d);
  if (st != EG_MLA_OK) return st;
  if (n_tokens < 0 || hidden < 1 || num_slots < 0) return EG_MLA_ERR_INVALID_ARG;
  if (hidden > 32768) return EG_MLA_ERR_UNSUPPORTED;  // x row staged in LDS
  if (d->rope_dim % 2 != 0) return EG_MLA_ERR_INVALID_ARG;
  if (n_tokens == 0) return EG_MLA_OK;
  if (!x || !token_ids || !positions || !slots || !w_dkv || !latent_cache || !token_id_cache)
    return EG_MLA_ERR_INVALID_ARG;
  return EG_MLA_OK;
}

eg_mla_status validate_gate_rows(const eg_mla_dims* d, int32_t emb_dim, int32_t emb_vocab, int64_t n,
                                 const int32_t* ids, const void* emb, const void* w_ue, const void* out) {
  eg_mla_status st = check_dims(d);
  if (st != EG_MLA_OK) return st;
  if (emb_dim < 1 || emb_vocab < 1 || n < 0) return EG_MLA_ERR_INVALID_ARG;
  if (emb_dim > 16384) return EG_MLA_ERR_UNSUPPORTED;  // one embedding row staged in LDS (VALU kernel)
  if (n == 0) return EG_MLA_OK;
  if (!ids || !emb || !w_ue || !out) return EG_MLA_ERR_INVALID_ARG;
  return EG_MLA_OK;
}

size_t prefill_workspace_bytes(const eg_mla_dims& d, int32_t seq_len) {
  const size_t T = static_cast<size_t>(std::max(seq_len, 0));
  const size_t H = static_cast<size_t>(d.num_heads);
  // fp32 explicit keys [H, T, d_h + d_r] and values [H, T, d_v]
  size_t k = align_up(H * T * static_cast<size_t>(d.head_dim + d.rope_dim) * 4);
  size_t v = align_up(H * T * static_cast<size_t>(d.v_head_dim) * 4);
  return std::max<size_t>(k + v, kAlign);
}

eg_mla_status validate_prefill(const eg_mla_dims* d, int32_t seq_len, const void* q, const void* latent,
                               const int32_t* token_ids, const void* gate_table, const void* w_uk,
                               const void* w_uv, const void* workspace, size_t workspace_bytes,
                               const void* out) {
  eg_mla_status st = check_dims(d);
  if (st != EG_MLA_OK) return st;
  if (seq_len < 0) return EG_MLA_ERR_INVALID_ARG;
  if (seq_len > 32768) return EG_MLA_ERR_UNSUPPORTED;  // one score row staged in LDS
  if (seq_len == 0) return EG_MLA_OK;
  if (!q || !latent || !token_ids || !gate_table || !w_uk || !w_uv || !out) return EG_MLA_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < prefill_workspace_bytes(*d, seq_len)) return EG_MLA_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return EG_MLA_ERR_WORKSPACE;
  return EG_MLA_OK;
}

bool prefill_varlen_absorbed(const eg_mla_dims& d) {
  return d.dtype == EG_MLA_BF16 && d.num_heads == 16 && d.head_dim == 128 && d.v_head_dim == 128 &&
         d.latent_dim == 128 && d.rope_dim == 64 && d.gate_dim == d.latent_dim;
}

bool prefill_varlen_shape_ok(const eg_mla_dims& d) {
  if (prefill_varlen_absorbed(d)) return true;
  // the explicit form: any head count, d_c a multiple of 64
  return d.dtype == EG_MLA_BF16 && d.head_dim == 128 && d.v_head_dim == 128 && d.rope_dim == 64 &&
         d.latent_dim % 64 == 0 && d.gate_dim == d.latent_dim;
}

PrefillVarlenLayout prefill_varlen_layout(const eg_mla_dims& d, int32_t total_tokens) {
  const size_t T = static_cast<size_t>(std::max(total_tokens, 0));
  const size_t H = static_cast<size_t>(d.num_heads);
  PrefillVarlenLayout L;
  L.off_seq_start = 0;  // int32 [T]
  if (prefill_varlen_absorbed(d)) {
    L.off_qf = align_up(T * 4);                                                                    // fp16 | bf16 [T][H][d_c + d_r]
    L.off_olat = L.off_qf + align_up(T * H * static_cast<size_t>(d.latent_dim + d.rope_dim) * 2);  // fp16 [T][H][d_c]
    L.off_ct = L.off_olat + align_up(T * H * static_cast<size_t>(d.latent_dim) * 2);             // fp16 [T][d_c]
    L.bytes = std::max<size_t>(L.off_ct + align_up(T * static_cast<size_t>(d.latent_dim) * 2), kAlign);
  } else {
    L.off_qf = align_up(T * 4);                                                  // K^C: fp16 [H][T][d_h]
    L.off_olat = L.off_qf + align_up(T * H * static_cast<size_t>(d.head_dim) * 2);  // V: fp16 [H][T][d_v]
    L.off_ct = L.off_olat + align_up(T * H * static_cast<size_t>(d.v_head_dim) * 2);  // bf16 hi, lo [2][T][d_c]
    L.bytes = std::max<size_t>(L.off_ct + 2 * align_up(T * static_cast<size_t>(d.latent_dim) * 2), kAlign);
  }
  return L;
}

eg_mla_status validate_prefill_varlen(const eg_mla_dims* d, int32_t batch, int32_t total_tokens,
                                      const int32_t* cu_seqlens, const void* q, const void* latent,
                                      const int32_t* token_ids, const void* gate_table, const void* w_uk,
                                      const void* w_uv, const void* workspace, size_t workspace_bytes,
                                      const void* out) {
  eg_mla_status st = check_dims(d);
  if (st != EG_MLA_OK) return st;
  if (batch < 1 || total_tokens < 0) return EG_MLA_ERR_INVALID_ARG;
  if (!prefill_varlen_shape_ok(*d)) return EG_MLA_ERR_UNSUPPORTED;
  if (total_tokens == 0) return EG_MLA_OK;
  if (!cu_seqlens || !q || !latent || !token_ids || !gate_table || !w_uk || !w_uv || !out)
    return EG_MLA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(latent) || !aligned16(gate_table) || !aligned16(w_uk) || !aligned16(w_uv) ||
      !aligned16(out))
    return EG_MLA_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < prefill_varlen_layout(*d, total_tokens).bytes) return EG_MLA_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return EG_MLA_ERR_WORKSPACE;
  return EG_MLA_OK;
}

bool literal_tile_shape(const eg_mla_dims& d) {
  return d.dtype == EG_MLA_BF16 && d.latent_dim == 128 && d.head_dim == 128 && d.v_head_dim == 128 &&
         d.rope_dim == 64 && d.num_heads <= 160 && literal_lds_bytes(d.num_heads) <= 160 * 1024;
}

size_t literal_generic_lds_bytes(const eg_mla_dims& d) {
  // latents of a group of 8 tokens, key dots and weights [8][H], moment sums
  // [4][8][2], per-token figures [3][8], per-head sums [2][H] and softmax
  // state [3][H], value sums [H][d_v] (all fp32)
  const size_t H = static_cast<size_t>(d.num_heads);
  return 4 * (8 * static_cast<size_t>(d.latent_dim) + 16 * H + 64 + 24 + 5 * H +
              H * static_cast<size_t>(d.v_head_dim));
}

size_t literal_lds_bytes(int num_heads) {
  // weight / gate-tile region, per-wave scores [4][H][32], value sums [4][d_v],
  // two sums per head, per-wave figures per head, token means [4][32] (all fp32)
  return 272 * 256 + 4 * static_cast<size_t>(num_heads) * 32 * 4 + 4 * 128 * 4 +
         static_cast<size_t>(num_heads) * (2 + 12) * 4 + 4 * 32 * 4;
}

size_t literal_workspace_bytes(const eg_mla_dims& d, int32_t batch, int32_t max_pages_per_seq) {
  const int64_t cap = static_cast<int64_t>(std::max(max_pages_per_seq, 0)) * d.page_size;
  const int64_t tiles = (cap + 127) / 128;
  return std::max<size_t>(align_up(static_cast<size_t>(std::max(batch, 0)) * static_cast<size_t>(tiles) *
                                   d.num_heads * (d.v_head_dim + 4) * sizeof(float)),
                          kAlign);
}

eg_mla_status validate_literal(const eg_mla_dims* d, int32_t batch, const void* q, const void* latent_cache,
                               const int32_t* token_id_cache, const void* gate_full, const void* w_uk,
                               const void* w_uv, const void* ln_w, const void* ln_b, uint32_t flags,
                               const int32_t* seq_lens, const int32_t* page_table, int32_t max_pages_per_seq,
                               int64_t num_slots, const void* workspace, size_t workspace_bytes, const void* out) {
  eg_mla_status st = check_dims(d);
  if (st != EG_MLA_OK) return st;
  if (batch < 0 || max_pages_per_seq < 0 || num_slots < 0) return EG_MLA_ERR_INVALID_ARG;
  if ((flags & ~(EG_MLA_LITERAL_NO_LN | EG_MLA_LITERAL_ADD)) != 0) return EG_MLA_ERR_INVALID_ARG;
  if (literal_tile_shape(*d)) {
    // gate rows are addressed by 32-bit byte offsets in the tile kernel
    if (static_cast<int64_t>(d->vocab_size) * d->num_heads * (d->head_dim + d->v_head_dim) * 2 >=
        (int64_t{1} << 32))
      return EG_MLA_ERR_UNSUPPORTED;
  } else if (literal_generic_lds_bytes(*d) > 160 * 1024) {
    return EG_MLA_ERR_UNSUPPORTED;  // the generic kernel's tile state does not fit in LDS
  }
  if (static_cast<int64_t>(max_pages_per_seq) * d->page_size > (int64_t{1} << 30)) return EG_MLA_ERR_UNSUPPORTED;
  if (num_slots >= (int64_t{1} << 31)) return EG_MLA_ERR_UNSUPPORTED;
  if (batch == 0) return EG_MLA_OK;
  if (!q || !gate_full || !w_uk || !w_uv || !seq_lens || !out || !latent_cache || !token_id_cache)
    return EG_MLA_ERR_INVALID_ARG;
  if (max_pages_per_seq < 1 || num_slots < 1) return EG_MLA_ERR_INVALID_ARG;
  if (!page_table && static_cast<int64_t>(batch) * max_pages_per_seq * d->page_size > num_slots)
    return EG_MLA_ERR_INVALID_ARG;  // contiguous rows: every sequence's capacity must fit in the cache
  if ((flags & EG_MLA_LITERAL_NO_LN) == 0 && (!ln_w || !ln_b)) return EG_MLA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(latent_cache) || !aligned16(gate_full) || !aligned16(w_uk) || !aligned16(w_uv))
    return EG_MLA_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < literal_workspace_bytes(*d, batch, max_pages_per_seq))
    return EG_MLA_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return EG_MLA_ERR_WORKSPACE;
  return EG_MLA_OK;
}

}  // namespace egmla

extern "C" {

const char* eg_mla_status_string(eg_mla_status s) {
  switch (s) {
    case EG_MLA_OK: return "EG_MLA_OK";
    case EG_MLA_ERR_INVALID_ARG: return "EG_MLA_ERR_INVALID_ARG: invalid argument";
    case EG_MLA_ERR_UNSUPPORTED: return "EG_MLA_ERR_UNSUPPORTED: shape or option not supported";
    case EG_MLA_ERR_WORKSPACE: return "EG_MLA_ERR_WORKSPACE: workspace missing, misaligned or too small";
    case EG_MLA_ERR_HIP: return "EG_MLA_ERR_HIP: HIP runtime or launch failure";
  }
  return "EG_MLA_ERR_UNKNOWN";
}

eg_mla_status eg_mla_check_dims(const eg_mla_dims* dims) { return egmla::check_dims(dims); }

size_t eg_mla_decode_workspace_size(const eg_mla_dims* dims, int32_t batch, int32_t max_pages_per_seq,
                                    const eg_mla_plan* plan) {
  if (egmla::check_dims(dims) != EG_MLA_OK || batch < 0 || max_pages_per_seq < 0) return 0;
  egmla::DecodePlan p;
  if (egmla::make_decode_plan(*dims, batch, max_pages_per_seq, plan, &p) != EG_MLA_OK) return 0;
  return p.bytes;
}

size_t eg_mla_prefill_workspace_size(const eg_mla_dims* dims, int32_t seq_len) {
  if (egmla::check_dims(dims) != EG_MLA_OK || seq_len < 0) return 0;
  return egmla::prefill_workspace_bytes(*dims, seq_len);
}

size_t eg_mla_prefill_varlen_workspace_size(const eg_mla_dims* dims, int32_t total_tokens) {
  if (egmla::check_dims(dims) != EG_MLA_OK || total_tokens < 0 || !egmla::prefill_varlen_shape_ok(*dims)) return 0;
  return egmla::prefill_varlen_layout(*dims, total_tokens).bytes;
}

}  // extern "C"
