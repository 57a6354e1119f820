/*
 * eg_mla.h -- C ABI of the EG-MLA decode library for AMD Instinct MI355X (gfx950).
 *
 * EG-MLA (Embedding-Gated Multi-head Latent Attention, arXiv 2509.16686)
 * caches one compressed latent c_t (d_c values, Sec. 3.1 Eq. (1)) and one
 * decoupled RoPE key k^R_t (d_r values shared by all heads, App. C
 * Eq. (C.10)) per token, plus the token's id i_t.  Each cached latent is
 * modulated by a token-specific gate g_t looked up from the token id
 * (Sec. 3.1 Eq. (3)-(5)).  This library applies the gate in the latent
 * space, c~_t = c_t * G[i_t], where G = Emb W^UE^T is the gate table folded
 * offline (the table-lookup variant of Sec. 5.2), so the per-head key and
 * value up-projections can be absorbed:
 *
 *   q_lat[h]  = W_UK[h]^T q^C[h]
 *   s[h,j]    = tau * (q_lat[h] . c~_j + q^R[h] . k^R_j),  tau = 1/sqrt(d_h + d_r)
 *   out[h]    = W_UV[h] * sum_j softmax_j(s[h,:]) c~_j
 *
 * which equals App. C Eq. (C.11)-(C.13) with k_{j,h} = [W_UK[h] c~_j ; k^R_j]
 * and v_{j,h} = W_UV[h] c~_j.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every tensor argument is a DEVICE pointer owned by the caller,
 *    row-major and contiguous.  The library never allocates or frees device
 *    memory and keeps no state between calls except cached device
 *    properties and the scratch array of eg_mla_decode_noalloc (a static
 *    device array of EG_MLA_NOALLOC_SCRATCH_BYTES per GPU).
 *  - Floating-point tensors have the storage type dims->dtype: IEEE fp32, or
 *    bf16 (16-bit brain float).  Arithmetic is fp32 (bf16 MFMA products with
 *    fp32 accumulation on the bf16 fast path).  Integer tensors are int32.
 *  - Weights follow the [out, in] convention of a linear layer: W_UK[h] is
 *    [d_h, d_c] (k^C = W_UK[h] c~), W_UV[h] is [d_v, d_c].
 *  - `stream` is a hipStream_t (NULL = the null stream).  Calls only enqueue
 *    work on it and return; they are safe to issue concurrently on
 *    different streams with disjoint workspaces.
 *  - Host-detectable errors (bad dims, null pointers, workspace too small)
 *    are returned before anything is enqueued.  A failed launch returns
 *    EG_MLA_ERR_HIP.  Device-side data are made safe rather than checked:
 *    sequence lengths are clamped to [0, capacity], token ids to [0, V),
 *    page numbers and slots to the cache; append skips out-of-range slots.
 */
#ifndef EG_MLA_H
#define EG_MLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum eg_mla_status {
  EG_MLA_OK = 0,
  EG_MLA_ERR_INVALID_ARG = 1,  /* null pointer, non-positive size, inconsistent dims */
  EG_MLA_ERR_UNSUPPORTED = 2,  /* valid but not implemented (e.g. gate_dim != latent_dim, forced path unavailable) */
  EG_MLA_ERR_WORKSPACE = 3,    /* workspace pointer null or smaller than the *_workspace_size query */
  EG_MLA_ERR_HIP = 4           /* a HIP launch or runtime call failed */
} eg_mla_status;

typedef enum eg_mla_dtype { EG_MLA_FP32 = 0, EG_MLA_BF16 = 1 } eg_mla_dtype;

/* Layer shapes.  gate_dim must equal latent_dim (the gate multiplies the
 * latent element-wise, Eq. (5) in the latent reading).  softmax_scale <= 0
 * selects 1/sqrt(head_dim + rope_dim) (App. C Eq. (C.13)). */
typedef struct eg_mla_dims {
  int32_t num_heads;    /* H   */
  int32_t head_dim;     /* d_h: non-RoPE part of each query/key head */
  int32_t v_head_dim;   /* d_v */
  int32_t latent_dim;   /* d_c */
  int32_t rope_dim;     /* d_r (may be 0) */
  int32_t gate_dim;     /* must equal d_c */
  int32_t vocab_size;   /* V: rows of the gate table */
  int32_t page_size;    /* P: tokens per cache page */
  float softmax_scale;  /* <= 0: default */
  int32_t dtype;        /* eg_mla_dtype of every floating-point tensor */
} eg_mla_dims;

/* Optional execution plan for eg_mla_decode_planned (tuning and tests). */
typedef enum eg_mla_path {
  EG_MLA_PATH_AUTO = 0,  /* MFMA when dtype is bf16 and the shape has a fast kernel, else VALU */
  EG_MLA_PATH_VALU = 1,  /* fp32 vector-ALU kernel, any shape and dtype */
  EG_MLA_PATH_MFMA = 2   /* bf16 matrix-core kernel; EG_MLA_ERR_UNSUPPORTED if the shape has none */
} eg_mla_path;

typedef struct eg_mla_plan {
  int32_t path;          /* eg_mla_path */
  int32_t split_tokens;  /* tokens per split-K work item, multiple of 32; 0 = automatic */
  /* Optional hipEvent_t handles (NULL = none) that time the token-streaming
   * split kernel alone with hipEventElapsedTime.  On the MFMA path they are
   * passed to hipExtLaunchKernelGGL and stamped by the dispatch itself (kernel
   * start and end); on the VALU path they are recorded on the call's stream
   * immediately before and after the kernel. */
  void* split_start_event;
  void* split_stop_event;
  /* Token-id slices per context split on the MFMA path with d_c = 128 and
   * d_r = 64: 0 = automatic (currently none), 1 = none, 8 = eight work items
   * per split, the one run by work-group x taking the tokens whose id is
   * x mod 8, so that each of the 8 XCDs gathers one eighth of the gate
   * table.  Other values: EG_MLA_ERR_INVALID_ARG; ignored by the other
   * kernels. */
  int32_t id_slices;
} eg_mla_plan;

/* Human-readable name of a status code (static string, never NULL). */
const char* eg_mla_status_string(eg_mla_status status);

/* Validates `dims` on the host.  EG_MLA_OK, EG_MLA_ERR_INVALID_ARG or
 * EG_MLA_ERR_UNSUPPORTED.  Touches no device. */
eg_mla_status eg_mla_check_dims(const eg_mla_dims* dims);

/* ---------------------------------------------------------------------------
 * Append: write new tokens into the latent cache (Sec. 3.1 Eq. (1); App. C
 * Eq. (C.10)).  For token i:
 *   [c | r]  = W_DKV x_i                      (W_DKV = [W^DKV ; W^KR], [d_c+d_r, hidden])
 *   c        = c / sqrt(mean(c^2) + 1e-6) * kv_norm_w      (only if kv_norm_w != NULL)
 *   k^R      = RoPE(r, positions[i])         (adjacent pairs (2m, 2m+1), angle pos*theta^(-2m/d_r))
 *   latent_cache[slots[i]] = [c | k^R]  (rounded to the storage type)
 *   token_id_cache[slots[i]] = token_ids[i]
 *
 *   x          [n_tokens, hidden]
 *   token_ids  [n_tokens] int32;  positions [n_tokens] int32 (0-based)
 *   slots      [n_tokens] int32 destination rows (page*P + offset); rows
 *              outside [0, num_slots) are skipped.  Duplicate slots race.
 *   w_dkv      [d_c + d_r, hidden];  kv_norm_w [d_c] or NULL
 *   latent_cache [num_slots, d_c + d_r];  token_id_cache [num_slots] int32
 * rope_theta <= 0 selects 10000.  n_tokens == 0 is a no-op.
 * ------------------------------------------------------------------------- */
eg_mla_status eg_mla_append(const eg_mla_dims* dims, int32_t n_tokens, int32_t hidden, const void* x,
                            const int32_t* token_ids, const int32_t* positions, const int32_t* slots,
                            const void* w_dkv, const void* kv_norm_w, float rope_theta, void* latent_cache,
                            int32_t* token_id_cache, int64_t num_slots, void* stream);

/* ---------------------------------------------------------------------------
 * Append with a workspace: the same operation and arguments as eg_mla_append
 * (Sec. 3.1 Eq. (1); App. C Eq. (C.10)), the same rows and ids.  With bf16
 * storage, d_r = 64, hidden a multiple of 256 and either d_c = 128 with
 * 1..2048 tokens or d_c = 512 with 1..2^20 tokens, W_DKV x_i is formed in
 * two passes: the hidden dimension is cut into S slices (S divides
 * hidden/256; many for few tokens, so that W_DKV spreads over many
 * work-groups, down to 1 for many tokens), pass 1 stores the fp32 partial
 * sums per slice in the workspace ([S, n_tokens, d_c + d_r]), pass 2 adds
 * them in slice order, applies the RMSNorm and RoPE and writes the rows.  Any
 * other call runs eg_mla_append (the workspace is not touched).
 *
 *   workspace  at least eg_mla_append_workspace_size(dims, n_tokens, hidden)
 *              bytes, 256-byte aligned, no initialisation needed; calls that
 *              share it must be ordered.  Too small or misaligned:
 *              EG_MLA_ERR_WORKSPACE before any launch.
 * eg_mla_append_workspace_size returns 0 for invalid dims or sizes.
 * ------------------------------------------------------------------------- */
size_t eg_mla_append_workspace_size(const eg_mla_dims* dims, int32_t n_tokens, int32_t hidden);

eg_mla_status eg_mla_append_ws(const eg_mla_dims* dims, int32_t n_tokens, int32_t hidden, const void* x,
                               const int32_t* token_ids, const int32_t* positions, const int32_t* slots,
                               const void* w_dkv, const void* kv_norm_w, float rope_theta, void* latent_cache,
                               int32_t* token_id_cache, int64_t num_slots, void* workspace,
                               size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Decode: one query row per sequence against its whole cached context
 * (App. C Eq. (C.13) with t = the current token; the gate of Eq. (3)-(5)
 * applied to each cached latent through its token id).
 *
 *   q             [B, H, d_h + d_r]   (q^C | q^R); q^R already rotated
 *   latent_cache  [num_slots, d_c + d_r]   (latent | RoPE key) per cached token
 *   token_id_cache[num_slots] int32   token id of every cached row
 *   gate_table    [V, d_c]            folded gate G = Emb W^UE^T
 *   w_uk          [H, d_h, d_c];  w_uv [H, d_v, d_c]
 *   seq_lens      [B] int32  cached tokens per sequence, current token
 *                 included; clamped to [0, max_pages_per_seq * P]; 0 gives zeros
 *   page_table    [B, max_pages_per_seq] int32, or NULL for contiguous
 *                 storage where token j of sequence b is row
 *                 b * max_pages_per_seq * P + j
 *   workspace     device scratch of at least
 *                 eg_mla_decode_workspace_size(dims, B, max_pages_per_seq, plan)
 *                 bytes, 256-byte aligned; contents need no initialisation
 *   out           [B, H, d_v]  in the storage type
 *
 * Arithmetic (bf16 storage, MFMA path): each gated latent is the exact fp32
 * product of two bf16 values rounded once to fp16, and the absorbed query
 * (fp32) is rounded once to fp16; the latent part of a score is one fp16
 * product accumulated in fp32, the RoPE part bf16 x bf16 (exact); the value
 * sum takes the fp16 gated latent and the probabilities rounded to fp16; the
 * split merge is fp32 and the up-projection takes the merged latent as bf16
 * hi + lo.  Queries, latents and their products must stay below 65504 in
 * magnitude (fp16's range).  The VALU path computes in fp32.  The call is asynchronous on `stream`; calls that share a
 * workspace must be ordered (same stream or synchronised).
 * ------------------------------------------------------------------------- */
size_t eg_mla_decode_workspace_size(const eg_mla_dims* dims, int32_t batch, int32_t max_pages_per_seq,
                                    const eg_mla_plan* plan /* NULL = automatic */);

eg_mla_status eg_mla_decode(const eg_mla_dims* dims, int32_t batch, const void* q, const void* latent_cache,
                            const int32_t* token_id_cache, const void* gate_table, const void* w_uk,
                            const void* w_uv, const int32_t* seq_lens, const int32_t* page_table,
                            int32_t max_pages_per_seq, int64_t num_slots, void* workspace,
                            size_t workspace_bytes, void* out, void* stream);

/* Same as eg_mla_decode with an explicit plan (NULL = automatic).  The
 * workspace must be sized with the same plan. */
eg_mla_status eg_mla_decode_planned(const eg_mla_dims* dims, int32_t batch, const void* q,
                                    const void* latent_cache, const int32_t* token_id_cache,
                                    const void* gate_table, const void* w_uk, const void* w_uv,
                                    const int32_t* seq_lens, const int32_t* page_table,
                                    int32_t max_pages_per_seq, int64_t num_slots, void* workspace,
                                    size_t workspace_bytes, void* out, void* stream, const eg_mla_plan* plan);

/* ---------------------------------------------------------------------------
 * Decode without a caller workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, arithmetic and automatic plan as
 * eg_mla_decode, minus the workspace: the call uses a scratch array of
 * EG_MLA_NOALLOC_SCRATCH_BYTES bytes that the library holds in device memory
 * (one per GPU, for as long as the process runs) and allocates nothing.
 *   - A call whose plan needs more than EG_MLA_NOALLOC_SCRATCH_BYTES of
 *     workspace (eg_mla_decode_workspace_size with a NULL plan) returns
 *     EG_MLA_ERR_WORKSPACE before anything is enqueued; so do the checks of
 *     eg_mla_decode (status codes as there).  32 MiB covers batch 32 at
 *     context 4096, batch 4 at 32768 and batch 256 at 2048 of the 16-head
 *     d_c = 128 layer, not the 128-head d_c = 512 one.
 *   - Every call on one GPU shares that GPU's array, which keeps the last
 *     call's contents (nothing in it needs to start at zero).  Calls that
 *     overlap on one GPU (different streams, or host threads without
 *     ordering) race: order them, or use eg_mla_decode with separate
 *     workspaces.
 *   - The first call on a device looks up the array's device address
 *     (hipGetSymbolAddress) with that device current; a failure of that
 *     lookup returns EG_MLA_ERR_HIP.
 * ------------------------------------------------------------------------- */
#define EG_MLA_NOALLOC_SCRATCH_BYTES (32u << 20)

eg_mla_status eg_mla_decode_noalloc(const eg_mla_dims* dims, int32_t batch, const void* q, const void* latent_cache,
                                    const int32_t* token_id_cache, const void* gate_table, const void* w_uk,
                                    const void* w_uv, const int32_t* seq_lens, const int32_t* page_table,
                                    int32_t max_pages_per_seq, int64_t num_slots, void* out, void* stream);

/* ---------------------------------------------------------------------------
 * Gate rows from the token embedding (Sec. 3.1 Eq. (3)-(4)): for i < n,
 *   out[i, :] = W^UE Emb[ids[i], :]
 * with e = emb_dim embedding components in and d_c = dims->latent_dim gate
 * values out, products accumulated in fp32 and rounded once to the storage
 * type (bf16 x bf16 MFMA products when dtype is bf16, emb_dim % 128 == 0,
 * d_c % 32 == 0, emb/w_ue 16-byte and out 8-byte aligned; fp32 VALU
 * otherwise).
 *   - ids = 0 .. V-1 gives the folded gate table G = Emb W^UE^T that
 *     eg_mla_decode takes (the table-lookup variant of Sec. 5.2, folded
 *     once when the model is loaded);
 *   - the ids of a step's cached tokens give the unfolded model's gates for
 *     that step; eg_mla_decode then takes `out` as its gate table with a
 *     token_id_cache that holds, for each cached row, its row index in `out`
 *     (dims->vocab_size = n).
 *
 *   emb   [emb_vocab, emb_dim];  w_ue [d_c, emb_dim] ([out, in]);
 *   ids   [n] int32, clamped to [0, emb_vocab);  out [n, d_c]
 * n == 0 is a no-op.  emb_dim above 16384 is EG_MLA_ERR_UNSUPPORTED.
 * ------------------------------------------------------------------------- */
eg_mla_status eg_mla_gate_rows(const eg_mla_dims* dims, int32_t emb_dim, int32_t emb_vocab, int64_t n,
                               const int32_t* ids, const void* emb, const void* w_ue, void* out, void* stream);

/* ---------------------------------------------------------------------------
 * Gate rows of the distinct ids of a step (Sec. 3.1 Eq. (3)-(4)): for every
 * id among ids[0 .. n),
 *   table[id, :] = W^UE Emb[id, :]
 * with the arithmetic of eg_mla_gate_rows (the same bits); rows of ids not
 * in the list are left as they are.  This is the unfolded model's gate
 * computation with each distinct id computed once: eg_mla_decode then takes
 * `table` as its gate table with the step's own token ids
 * (dims->vocab_size = emb_vocab).  On the MFMA path a first kernel claims
 * each id with an atomic exchange of `stamp` into `marks` and lists the ids
 * whose claim found another value; the gate rows are computed over that
 * list only.  Other paths compute every row and store identical bits for
 * repeated ids.
 *
 *   emb, w_ue, ids as for eg_mla_gate_rows;  table [emb_vocab, d_c]
 *   marks  device workspace of eg_mla_gate_table_marks_size(dims, emb_dim,
 *          emb_vocab) bytes (a 128-byte stamp line per id, two counters, an
 *          id list),
 *          4-byte aligned, owned by the caller: zero it before the first
 *          call and keep it between calls;
 *   stamp  1 on the first call after the marks were zeroed, then the previous
 *          call's stamp plus one (the counters alternate by the stamp's
 *          parity); zero the marks again before the stamp would wrap to 0.
 * Calls that share marks must be ordered (same stream or synchronised).
 * n == 0 is a no-op (the stamp is not consumed: the next call takes it);
 * stamp == 0 is EG_MLA_ERR_INVALID_ARG; marks null, misaligned or smaller
 * than the query is EG_MLA_ERR_WORKSPACE.
 * eg_mla_gate_table_marks_size returns 0 for invalid dims or sizes.
 * ------------------------------------------------------------------------- */
size_t eg_mla_gate_table_marks_size(const eg_mla_dims* dims, int32_t emb_dim, int32_t emb_vocab);

eg_mla_status eg_mla_gate_table(const eg_mla_dims* dims, int32_t emb_dim, int32_t emb_vocab, int64_t n,
                                const int32_t* ids, const void* emb, const void* w_ue, void* table, void* marks,
                                size_t marks_bytes, uint32_t stamp, void* stream);

/* ---------------------------------------------------------------------------
 * Prefill reference: plain causal attention over one sequence of T tokens in
 * the explicit (non-absorbed) form of App. C Eq. (C.2), (C.6), (C.11)-(C.13):
 * it materialises k_{j,h} = [W_UK[h] c~_j ; k^R_j] and v_{j,h} = W_UV[h] c~_j
 * in fp32 in the workspace and runs one softmax per (t, h) over j <= t.
 * A plain second implementation for cross-checks, not a fast prefill.
 *
 *   q [T, H, d_h + d_r];  latent [T, d_c + d_r];  token_ids [T] int32
 *   gate_table, w_uk, w_uv as for decode;  out [T, H, d_v]
 * ------------------------------------------------------------------------- */
size_t eg_mla_prefill_workspace_size(const eg_mla_dims* dims, int32_t seq_len);

eg_mla_status eg_mla_prefill_ref(const eg_mla_dims* dims, int32_t seq_len, const void* q, const void* latent,
                                 const int32_t* token_ids, const void* gate_table, const void* w_uk,
                                 const void* w_uv, void* workspace, size_t workspace_bytes, void* out,
                                 void* stream);

/* ---------------------------------------------------------------------------
 * Causal prefill of a batch of sequences packed back to back (App. C
 * Eq. (C.2), (C.11)-(C.13) in the absorbed form, with the latent-space gate of
 * Sec. 3.1 Eq. (3)-(5)): row (t, h) attends to the tokens j <= t of t's own
 * sequence,
 *   out[t,h] = W_UV[h] sum_j softmax_j(tau (q_lat[t,h].c~_j + q^R[t,h].k^R_j)) c~_j,
 *   q_lat[t,h] = W_UK[h]^T q^C[t,h],  c~_j = c_j (.) G[token_ids[j]].
 * MFMA kernels for bf16 storage with d_h = d_v = 128 and d_r = 64: the
 * absorbed form for d_c = 128 with 16 heads (all heads share the gated latent
 * as key and value), the explicit form of App. C Eq. (C.2), (C.6) for any
 * other head count and d_c a multiple of 64 (K^C = W_UK[h] c~ and
 * V = W_UV[h] c~ per head, then attention per head; 3.4x fewer flops per pair
 * than the absorbed form at d_c 512).  Other shapes: EG_MLA_ERR_UNSUPPORTED
 * (eg_mla_prefill_ref covers any shape, one sequence at a time).  The matrix
 * products take fp16 operands for the latent parts (values below 65504 in
 * magnitude) and bf16 ones for the RoPE parts.
 *
 *   cu_seqlens [batch + 1] int32 (device): sequence b is tokens
 *       cu_seqlens[b] .. cu_seqlens[b+1]-1; cu_seqlens[0] = 0,
 *       non-decreasing, cu_seqlens[batch] = total_tokens (empty sequences
 *       allowed).  Values outside that are not checked; the kernels clamp
 *       every index into range.
 *   q [total, H, d_h + d_r] (q^R already rotated); latent [total, d_c + d_r]
 *       (rows as eg_mla_append writes them); token_ids [total];
 *   gate_table, w_uk, w_uv as for decode;  out [total, H, d_v].
 *   workspace: eg_mla_prefill_varlen_workspace_size bytes, 256-byte aligned
 *       (per-token sequence starts; absorbed form: the absorbed queries
 *       [T][H][d_c + d_r] (q_lat fp16, q^R bf16), the normalised latent
 *       outputs in fp16 [T][H][d_c] and the gated latents in fp16 [T][d_c];
 *       explicit form: K^C and V in fp16, [H][T][128] each, and the gated
 *       latents as bf16 hi and lo rows, [T][d_c] each).
 * Pointers 16-byte aligned.  total_tokens == 0 is a no-op.
 * ------------------------------------------------------------------------- */
size_t eg_mla_prefill_varlen_workspace_size(const eg_mla_dims* dims, int32_t total_tokens);

eg_mla_status eg_mla_prefill_varlen(const eg_mla_dims* dims, int32_t batch, int32_t total_tokens,
                                    const int32_t* cu_seqlens, const void* q, const void* latent,
                                    const int32_t* token_ids, const void* gate_table, const void* w_uk,
                                    const void* w_uv, void* workspace, size_t workspace_bytes, void* out,
                                    void* stream);

/* ---------------------------------------------------------------------------
 * Decode with the paper-literal gate (Sec. 3.1 Eq. (2)-(5) as printed and the
 * model listing's order): for every cached token j of sequence b,
 *   kv_j = [W_UK[h] c_j ; W_UV[h] c_j]_h      (W^UKV c_j, head-major, H (d_h + d_v) dims)
 *   x_j  = kv_j (.) G[i_j]     (or kv_j + G[i_j] with EG_MLA_LITERAL_ADD)
 *   y_j  = LN(x_j)             over all H (d_h + d_v) dims, eps 1e-5, weight and
 *                              bias (skipped with EG_MLA_LITERAL_NO_LN)
 * and per head out[b,h] = sum_j softmax_j(tau q_h . [y_j[h,:d_h] ; k^R_j]) y_j[h,d_h:].
 * The gate follows the up-projection and the LayerNorm spans all heads, so
 * nothing is absorbed: each call up-projects every cached token.  (The main
 * decode applies the gate to the latent; this call is the literal variant
 * and its two ablations.)
 *
 * The MFMA tile kernel takes bf16 storage with d_c = d_h = d_v = 128,
 * d_r = 64, at most 160 heads and a gate table below 4 GB (32-bit row
 * offsets).  Every other layer (any d_c, d_h, d_v, d_r, bf16 or fp32
 * storage) takes a generic kernel of the same arithmetic, plain fp32 and not
 * tuned, while its per-tile state fits the LDS: 4 (8 d_c + H (d_v + 21) + 88)
 * bytes <= 160 KB (the 128-head d_c 512 layer fits); beyond that
 * EG_MLA_ERR_UNSUPPORTED.  dims->gate_dim is not used here (it must still
 * pass eg_mla_check_dims).  Softmax partials are formed per 128-token tile
 * and merged, so the context length is not limited.
 *
 *   q, latent_cache, token_id_cache, w_uk, w_uv, seq_lens, page_table,
 *       max_pages_per_seq, num_slots: as for eg_mla_decode;
 *   gate_full [vocab_size, H (d_h + d_v)]: per-token gate rows, head-major
 *       like kv (per head d_h key dims, then d_v value dims);
 *   ln_weight, ln_bias [H (d_h + d_v)] (may be null with EG_MLA_LITERAL_NO_LN);
 *   flags: 0, EG_MLA_LITERAL_NO_LN, EG_MLA_LITERAL_ADD or both;
 *   workspace: eg_mla_decode_literal_workspace_size(dims, batch,
 *       max_pages_per_seq) bytes, 256-byte aligned (fp32 softmax partials
 *       per sequence, 128-token tile and head);  out [batch, H, d_v].
 * Host-detectable errors as for eg_mla_decode.
 * ------------------------------------------------------------------------- */
#define EG_MLA_LITERAL_NO_LN 1u
#define EG_MLA_LITERAL_ADD 2u

size_t eg_mla_decode_literal_workspace_size(const eg_mla_dims* dims, int32_t batch, int32_t max_pages_per_seq);

eg_mla_status eg_mla_decode_literal(const eg_mla_dims* dims, int32_t batch, const void* q, const void* latent_cache,
                                    const int32_t* token_id_cache, const void* gate_full, const void* w_uk,
                                    const void* w_uv, const void* ln_weight, const void* ln_bias, uint32_t flags,
                                    const int32_t* seq_lens, const int32_t* page_table, int32_t max_pages_per_seq,
                                    int64_t num_slots, void* workspace, size_t workspace_bytes, void* out,
                                    void* stream);

#ifdef __cplusplus
}
#endif

#endif /* EG_MLA_H */
