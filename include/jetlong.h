/*
 * jetlong.h -- C ABI of libjetlong.so: fused causal bifocal-RoPE attention
 * (Jet-Long, arXiv 2607.07740) for AMD Instinct MI355X (gfx950).
 *
 * The method (Sec. 3, Eq. (1)): a query at position q attends to a key at
 * position k <= q with the score
 *     <R(q) x_q, R(k) x_k>            if q - k <= w_local   (local view)
 *     <R(f(q)) x_q, R(f(k)) x_k>      if q - k >  w_local   (remote view)
 * where R(p) is the RoPE rotation to position p, f(x) = floor(x / G) (Eq. (3))
 * and G = max(1, ceil(L / w_pretrained)) (Eq. (2)) for the current length L.
 * The remote rotation is applied on the fly to raw (pre-RoPE) Q/K as the
 * correction rotation of Sec. 3.2 (Eqs. (5)-(6)); no rotated copy of K is ever
 * written.  Local and remote partial softmax states are merged by the
 * max-shifted, linear-space rule of Sec. 3.3, Eq. (7).
 *
 * Conventions shared by every entry point:
 *  - Tensors are DEVICE pointers to contiguous row-major storage; "bf16" is
 *    IEEE bfloat16 stored as 16-bit words.  Every tensor pointer must be
 *    16-byte aligned.  The caller owns all tensors and workspaces.
 *  - RoPE uses the rotate-half pairing (element i with i + head_dim/2) and
 *    frequencies omega_i = rope_theta^(-2i/head_dim); positions are 0-based;
 *    the softmax scale is 1/sqrt(head_dim).
 *  - Grouped-query attention: query head h reads kv head h / (Hq / Hkv).
 *  - head_dim must be 128 (other values return JL_ERR_UNSUPPORTED).
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream).  Arguments are validated on the host before anything is
 *    launched; on any error nothing is written and nothing is launched.
 *  - Where a call allocates or waits.  The library keeps per-device caches
 *    that a call may have to build or grow; only then does it allocate and
 *    wait, and a later call with the same or a smaller shape does neither:
 *      - the RoPE cos/sin table (per device and rope_theta, grown by
 *        doubling to cover the call's positions): every prefill and decode
 *        entry point; growing allocates and waits for `stream`;
 *      - the prefill scratch (per device and stream): jl_bifocal_prefill,
 *        jl_rope_attention, their _map, _chunk and _varlen forms; growing
 *        waits for `stream`, frees the old buffer and allocates;
 *      - the frequency-map table (one per device): jl_bifocal_prefill_map
 *        with JL_REMOTE_FREQ; a new (rope_theta, L, w_pretrained) waits for
 *        the whole device, then rebuilds the table in place, or in a buffer
 *        of at least twice the capacity when L does not fit.
 *    The literal and decode entry points use the caller's workspace and
 *    allocate nothing else.  jl_release_caches frees every cache.
 *  - Thread safety: calls may come from several host threads; the library's
 *    shared state (the caches above and the debug settings below) is guarded
 *    by mutexes.  Calls that share output buffers must be ordered by the
 *    caller.
 *  - Status codes are returned; no exception crosses the ABI and nothing
 *    aborts.  jl_last_error() gives a human-readable detail for the calling
 *    thread's most recent failure.
 */
#ifndef JETLONG_H
#define JETLONG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  JL_OK = 0,
  JL_ERR_INVALID_ARG = 1, /* bad shape, pointer, alignment or window value      */
  JL_ERR_UNSUPPORTED = 2, /* valid but not built (head_dim != 128, GQA group)   */
  JL_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required         */
  JL_ERR_HIP = 4          /* HIP runtime error (launch, allocation, no device)  */
};

/* Name of a status code ("JL_OK", ...); never NULL. */
const char* jl_status_string(int status);

/* Detail message of the calling thread's last failed call ("" if none). */
const char* jl_last_error(void);

/* ABI version: major * 10000 + minor * 100 + patch. */
int jl_version(void);

/*
 * Group size of Sec. 3.1, Eq. (2), computed on the host:
 * G = max(1, ceil(L / w_pretrained)).  Returns -1 if L < 1 or w_pretrained < 1.
 */
int64_t jl_group_size(int64_t L, int64_t w_pretrained);

/*
 * Bifocal prefill (Sec. 3, Eq. (1); merge of Sec. 3.3, Eq. (7)).
 *   q   bf16 [B, L, Hq, head_dim]   raw (pre-RoPE) queries, position = row index
 *   k   bf16 [B, L, Hkv, head_dim]  raw (pre-RoPE) keys
 *   v   bf16 [B, L, Hkv, head_dim]
 *   o   bf16 [B, L, Hq, head_dim]   output (written)
 *   lse fp32 [B, Hq, L] or NULL     natural-log softmax normaliser per row
 * One G for the whole call, from this call's L (all B sequences share L).
 * w_pretrained >= 1, w_local >= 0; keys with q - k <= w_local use the base
 * rotation, older keys the remote one.  When G == 1 the output equals
 * jl_rope_attention bit for bit (the method reduces to the base model).
 * Requires Hq % Hkv == 0, 256 % (Hq / Hkv) == 0 and B * Hkv <= 65535.
 * K is read raw: the keys of each 64-key tile are loaded into registers and
 * rotated to the view of the visit (R(k) x_k on the band, R(f(k)) x_k beyond
 * it, Sec. 3.2); the rotated tile is kept only in on-chip memory and no
 * rotated key is written anywhere.
 * Memory: V is transposed into a library-owned scratch buffer of
 * B * Hkv * ceil(L / 64) * 16 KB bytes of tile images plus
 * 4 * B * Hkv * L + 256 bytes for the list of blocks the checked pass reruns,
 * one per (device, stream), grown on demand (growing waits for the stream)
 * and freed by jl_release_caches; q, k, v are only read.
 */
int jl_bifocal_prefill(const void* q, const void* k, const void* v, void* o, float* lse, int B,
                       int Hq, int Hkv, int L, int head_dim, double rope_theta, int w_pretrained,
                       int w_local, void* stream);

/* Remote-view maps for jl_bifocal_prefill_map. */
enum {
  JL_REMOTE_ALIAS = 0, /* Eq. (3): remote positions f(x) = floor(x / G), base frequencies */
  JL_REMOTE_FREQ = 1   /* Sec. 4.5 / Table 6 ablation: positions kept, frequencies rescaled */
};

/*
 * jl_bifocal_prefill with a choice of remote view (Sec. 4.5, Table 6, the
 * ablation that replaces position aliasing by frequency interpolation).
 *   remote_map = JL_REMOTE_ALIAS  identical to jl_bifocal_prefill;
 *   remote_map = JL_REMOTE_FREQ   the remote view keeps each query and key at
 *     its own position and rotates it with rescaled frequencies omega'_i: with
 *     s = max(1, L / w_pretrained) and r_i = w_pretrained * omega_i / (2 pi) the
 *     number of turns pair i completes over the pretraining window,
 *     gamma_i = clamp((r_i - 1) / 31, 0, 1) and
 *     omega'_i = (1 - gamma_i) omega_i / s + gamma_i omega_i (YaRN's per-pair
 *     ramp, alpha = 1, beta = 32; no attention temperature).  The local window,
 *     the masks and the Eq. (7) merge are unchanged.
 * When L <= w_pretrained (s = 1, G = 1) both maps run the vanilla kernel.
 * The frequency map keeps one library-owned table of cos/sin(p * omega'_i),
 * L x 512 bytes per device, for the last (rope_theta, L, w_pretrained) used;
 * a new configuration waits for the whole device and rebuilds that table in
 * place (in a new buffer of at least twice the capacity when L does not fit,
 * the old one freed), then waits for the stream.  jl_release_caches frees it.
 * Other arguments, scratch and errors as in jl_bifocal_prefill; remote_map
 * outside {0, 1} -> JL_ERR_INVALID_ARG.
 */
int jl_bifocal_prefill_map(const void* q, const void* k, const void* v, void* o, float* lse,
                           int B, int Hq, int Hkv, int L, int head_dim, double rope_theta,
                           int w_pretrained, int w_local, int remote_map, void* stream);

/*
 * Continued (chunked) prefill over an existing raw cache (Sec. 3.2: the cache
 * keeps keys at base coordinates and is never rewritten when G changes).
 *   q       bf16 [B, n_queries, Hq, head_dim]  raw queries at positions
 *                                              q_start .. q_start + n_queries - 1
 *   k_cache bf16 [B, max_len, Hkv, head_dim]   raw keys; rows [0, q_start + n_queries)
 *   v_cache bf16 [B, max_len, Hkv, head_dim]   must hold the chunk's own keys too
 *   o       bf16 [B, n_queries, Hq, head_dim]  output (written)
 *   lse     fp32 [B, Hq, n_queries] or NULL
 * The call's sequence length is L = q_start + n_queries: G = max(1,
 * ceil(L / w_pretrained)) for every query of the chunk, as in a prefill of
 * length L, so the output equals rows q_start .. L - 1 of
 * jl_bifocal_prefill over the first L cache rows.  The caches are only read:
 * keys are rotated on chip per visit, as in jl_bifocal_prefill, and values
 * [0, L) are transposed into the library scratch, so a chunk costs O(L)
 * extra work on top of its attention.  Requires 0 <= q_start, n_queries >= 1,
 * q_start + n_queries <= max_len; other requirements and errors as in
 * jl_bifocal_prefill.
 */
int jl_bifocal_prefill_chunk(const void* q, const void* k_cache, const void* v_cache, void* o,
                             float* lse, int B, int Hq, int Hkv, int q_start, int n_queries,
                             int max_len, int head_dim, double rope_theta, int w_pretrained,
                             int w_local, void* stream);

/* The vanilla counterpart of jl_bifocal_prefill_chunk (base rotation only). */
int jl_rope_attention_chunk(const void* q, const void* k_cache, const void* v_cache, void* o,
                            float* lse, int B, int Hq, int Hkv, int q_start, int n_queries,
                            int max_len, int head_dim, double rope_theta, void* stream);

/*
 * jl_bifocal_prefill_chunk over paged caches (Sec. 3.2: the raw cache is
 * read, never rewritten, whatever G the chunk's length gives).
 *   k_pages, v_pages bf16 [n_pages, page_size, Hkv, head_dim] device pools
 *   block_table int32 [B, max_pages] (device): key x of sequence b is row
 *               x % page_size of page block_table[b][x / page_size]
 * The pages of keys [0, q_start + n_queries) must be written (the chunk's own
 * keys included); entries outside [0, n_pages) are clamped into the pool
 * (garbage in, no fault).  The output equals jl_bifocal_prefill_chunk's on a
 * dense cache holding the same rows, bit for bit.  page_size must be a power
 * of two, max_pages, n_pages >= 1, and q_start + n_queries <=
 * max_pages * page_size (else JL_ERR_INVALID_ARG); page_size < 64 (a page
 * must hold whole 64-key tiles) or more than 4096 pages per sequence (the
 * attention kernel keeps the list in LDS) -> JL_ERR_UNSUPPORTED.  q, o, lse,
 * scratch and the other arguments and errors as in jl_bifocal_prefill_chunk.
 */
int jl_bifocal_prefill_chunk_paged(const void* q, const void* k_pages, const void* v_pages,
                                   const int32_t* block_table, int max_pages, int page_size,
                                   int n_pages, void* o, float* lse, int B, int Hq, int Hkv,
                                   int q_start, int n_queries, int head_dim, double rope_theta,
                                   int w_pretrained, int w_local, void* stream);

/* The vanilla counterpart of jl_bifocal_prefill_chunk_paged. */
int jl_rope_attention_chunk_paged(const void* q, const void* k_pages, const void* v_pages,
                                  const int32_t* block_table, int max_pages, int page_size,
                                  int n_pages, void* o, float* lse, int B, int Hq, int Hkv,
                                  int q_start, int n_queries, int head_dim, double rope_theta,
                                  void* stream);

/*
 * Packed (variable-length) bifocal prefill: B independent sequences of
 * different lengths in one call, each computed exactly as jl_bifocal_prefill
 * would compute it alone -- its own L, G = max(1, ceil(L / w_pretrained))
 * (Eq. (2)), positions 0 .. L - 1, Eq. (3) remote positions and the Eq. (7)
 * bifocal result (a sequence with G = 1 gets the base model, as there).
 *   q, o: bf16 [total_tokens, Hq, head_dim]; k, v: bf16 [total_tokens, Hkv,
 *     head_dim] (raw, before RoPE); sequence s holds rows
 *     cu_seqlens[s] .. cu_seqlens[s + 1] - 1.
 *   lse: NULL or fp32 [Hq, total_tokens], natural-log row sums.
 *   cu_seqlens: DEVICE int32 [B + 1], non-decreasing from 0 to total_tokens
 *     (read by the kernels only; the call does not synchronise).
 *   max_seqlen: an upper bound of the sequence lengths; sets the RoPE table
 *     size.  Longer sequences are cut to their first max_seqlen rows.
 * Malformed cu_seqlens cannot cause an access outside the tensors: bounds are
 * clamped into [0, total_tokens] (a decreasing step gives an empty sequence)
 * and a sequence whose work would not fit the lists sized for well-formed
 * input is skipped; output rows of skipped, cut or uncovered positions are
 * left as they were.  Scratch (the library's, per stream): (Hkv *
 * (ceil(T / 64) + B)) V^T tile images of 16 KB plus two small work lists.  Other
 * requirements and errors as in jl_bifocal_prefill; only the Eq. (3) map.
 */
int jl_bifocal_prefill_varlen(const void* q, const void* k, const void* v, void* o, float* lse,
                              const int32_t* cu_seqlens, int B, int total_tokens, int max_seqlen,
                              int Hq, int Hkv, int head_dim, double rope_theta, int w_pretrained,
                              int w_local, void* stream);

/*
 * jl_bifocal_prefill_varlen with a choice of remote map (Sec. 4.5, Tab. 6),
 * as jl_bifocal_prefill_map offers it for one sequence.  JL_REMOTE_ALIAS is
 * jl_bifocal_prefill_varlen bit for bit; JL_REMOTE_FREQ gives every sequence
 * the frequency map of its own length: factor s = max(1, L / w_pretrained),
 * positions unchanged, each sequence equal bit for bit to jl_bifocal_prefill_map
 * on that sequence alone.  The per-sequence tables (768 bytes per token) are
 * built on the device into the library scratch.  Other arguments and errors
 * as in jl_bifocal_prefill_varlen; remote_map outside {0, 1} ->
 * JL_ERR_INVALID_ARG.
 */
int jl_bifocal_prefill_varlen_map(const void* q, const void* k, const void* v, void* o,
                                  float* lse, const int32_t* cu_seqlens, int B, int total_tokens,
                                  int max_seqlen, int Hq, int Hkv, int head_dim, double rope_theta,
                                  int w_pretrained, int w_local, int remote_map, void* stream);

/* The vanilla counterpart of jl_bifocal_prefill_varlen (base rotation only). */
int jl_rope_attention_varlen(const void* q, const void* k, const void* v, void* o, float* lse,
                             const int32_t* cu_seqlens, int B, int total_tokens, int max_seqlen,
                             int Hq, int Hkv, int head_dim, double rope_theta, void* stream);

/*
 * Vanilla causal RoPE attention with the same tiling and RoPE of raw Q/K at
 * base positions: the base model of Sec. 3 and the denominator of the
 * overhead measurements.  Arguments and scratch as in jl_bifocal_prefill.
 */
int jl_rope_attention(const void* q, const void* k, const void* v, void* o, float* lse, int B,
                      int Hq, int Hkv, int L, int head_dim, double rope_theta, void* stream);

/*
 * Bytes of device workspace jl_bifocal_prefill_literal needs for this shape:
 * 3 * B * L * Hq * head_dim * 4 (the window outputs) + the window LSEs
 * (3 * B * Hq * L * 4, rounded up to 256) + B * Hkv * ceil(L / 64) * 16 KB
 * (transposed value tiles) + 256 + 4 * B * Hkv * L (the window passes'
 * counters and list of query blocks for the checked rerun).  Returns 0 for
 * invalid arguments.
 */
size_t jl_prefill_literal_workspace_bytes(int B, int Hq, int Hkv, int L, int head_dim);

/*
 * Bifocal prefill with Eq. (7) of Sec. 3.3 taken literally: the three
 * attention calls A (band q - k <= w_local, base rotation), B (all causal
 * keys, remote rotation) and C (band, remote rotation) run as three calls
 * of the attention kernel (each as the fused call runs: a fast pass, then a
 * checked rerun of the blocks it lists), each
 * writing its normalised output O_X and its natural-log LSE_X, and a fourth
 * kernel merges them per row with
 *   M = max(LSE_A, LSE_B, LSE_C), W_X = exp(LSE_X - M),
 *   O = (W_A O_A + (W_B O_B - W_C O_C)) / (W_A + (W_B - W_C)),
 *   lse = M + ln(W_A + (W_B - W_C)),
 * in fp32.  This is the unfused variant the fused kernel of
 * jl_bifocal_prefill replaces; the two agree up to rounding, except where the
 * band dominates window B so strongly that the subtraction cancels (the
 * literal form loses precision there; the fused form does not subtract).
 * Arguments as in jl_bifocal_prefill, plus
 *   workspace, workspace_bytes: device memory of at least
 *     jl_prefill_literal_workspace_bytes(B, Hq, Hkv, L, head_dim) bytes,
 *     256-byte aligned, owned by the caller; contents on entry do not matter.
 *     On return (after the stream completes) it holds, for X = A, B, C
 *     (x = 0, 1, 2), O_X as fp32 [B, L, Hq, head_dim] at float offset
 *     x * B * L * Hq * head_dim, and LSE_X as fp32 [B, Hq, L] at float offset
 *     3 * B * L * Hq * head_dim + x * B * Hq * L.
 * When G == 1 the call runs the vanilla kernel, as jl_bifocal_prefill does,
 * with its transposed value tiles in the workspace's tile region; the window
 * outputs and LSEs are left unwritten.  Either way no library scratch is
 * used (only the RoPE table cache, as for every entry point).
 */
int jl_bifocal_prefill_literal(const void* q, const void* k, const void* v, void* o, float* lse,
                               int B, int Hq, int Hkv, int L, int head_dim, double rope_theta,
                               int w_pretrained, int w_local, void* workspace,
                               size_t workspace_bytes, void* stream);

/*
 * Bytes of device workspace the decode entry points need for this shape
 * (split-K partial softmax states).  Returns 0 for invalid arguments.
 */
size_t jl_decode_workspace_bytes(int B, int Hq, int Hkv, int max_len, int head_dim);

/*
 * Bifocal single-query decode on a raw KV cache (Sec. 3.2, Eqs. (4)-(6)).
 *   q        bf16 [B, Hq, head_dim]           raw new queries; the query of
 *                                              sequence b sits at position
 *                                              kv_lens[b] - 1
 *   k_cache  bf16 [B, max_len, Hkv, head_dim] raw (pre-RoPE) keys, the new
 *                                              token already appended
 *   v_cache  bf16 [B, max_len, Hkv, head_dim]
 *   kv_lens  int32 [B] DEVICE array, 1 <= kv_lens[b] <= max_len; positions
 *            at or past kv_lens[b] are never read.  The host cannot check
 *            it: a value below 1 is read as 1 and one past max_len as
 *            max_len, so a bad length gives wrong values, never an
 *            out-of-bounds read
 *   o        bf16 [B, Hq, head_dim] output (written)
 *   workspace, workspace_bytes: device scratch of at least
 *            jl_decode_workspace_bytes(B, Hq, Hkv, max_len, head_dim) bytes,
 *            16-byte aligned; its contents on entry do not matter.
 * G is taken per sequence from L = kv_lens[b] on the device, so one cache
 * serves every length and G change without being rewritten.
 * Requires Hq % Hkv == 0 and Hq / Hkv <= 8; max_len > 8388608 (2^23)
 * returns JL_ERR_UNSUPPORTED.
 */
int jl_bifocal_decode(const void* q, const void* k_cache, const void* v_cache,
                      const int32_t* kv_lens, int max_len, void* o, int B, int Hq, int Hkv,
                      int head_dim, double rope_theta, int w_pretrained, int w_local,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * jl_bifocal_decode for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments and results, bit for bit, without the
 * workspace: the split states and the fp32 cos/sin table live in one fixed
 * device array that the library holds on each device it runs on until the
 * process ends (88 MiB: the table of positions [0, 131072) and 24 MiB of
 * states).  No call allocates or frees device memory.
 *   max_len > 131072, or split states above 24 MiB
 *   (jl_decode_workspace_bytes(B, Hq, Hkv, max_len, 128) > 25165824)
 *     -> JL_ERR_UNSUPPORTED, checked on the host before any device work.
 * The first call on a device for a given rope_theta builds the table and
 * waits for it on `stream` (make that call outside graph capture); later
 * calls with that theta launch the two decode kernels only.  Every call on a
 * device shares that device's array, so calls that overlap on one device
 * (other streams, other threads) race; serialise them.  Other requirements
 * and errors as in jl_bifocal_decode.
 */
int jl_bifocal_decode_noalloc(const void* q, const void* k_cache, const void* v_cache,
                              const int32_t* kv_lens, int max_len, void* o, int B, int Hq,
                              int Hkv, int head_dim, double rope_theta, int w_pretrained,
                              int w_local, void* stream);

/* Vanilla RoPE decode with the same kernels (base rotation for every key). */
int jl_rope_attention_decode(const void* q, const void* k_cache, const void* v_cache,
                             const int32_t* kv_lens, int max_len, void* o, int B, int Hq,
                             int Hkv, int head_dim, double rope_theta, void* workspace,
                             size_t workspace_bytes, void* stream);

/*
 * Bytes of workspace jl_bifocal_decode_map needs: jl_decode_workspace_bytes,
 * for either remote map.  Returns 0 for invalid arguments.
 */
size_t jl_decode_map_workspace_bytes(int B, int Hq, int Hkv, int max_len, int head_dim,
                                     int remote_map);

/*
 * jl_bifocal_decode with a choice of remote map (the Sec. 4.5 / Tab. 6
 * ablation, as jl_bifocal_prefill_map does for prefill).
 *   remote_map  JL_REMOTE_ALIAS: identical to jl_bifocal_decode.
 *               JL_REMOTE_FREQ: remote pairs (q - k > w_local) keep their
 *               positions and rotate by omega'_i = (1 - gamma_i) omega_i / s +
 *               gamma_i omega_i (YaRN's ramp, alpha = 1, beta = 32, no
 *               temperature), with s = max(1, kv_lens[b] / w_pretrained) per
 *               sequence, so a ragged batch mixes factors the way it mixes G.
 *               Each workgroup forms the cos/sin rows it needs from its
 *               sequence's length (which lives on the device).
 *   workspace   at least jl_decode_map_workspace_bytes(..., remote_map) bytes,
 *               16-byte aligned, contents on entry irrelevant.
 * Other arguments, requirements and errors as in jl_bifocal_decode.
 */
int jl_bifocal_decode_map(const void* q, const void* k_cache, const void* v_cache,
                          const int32_t* kv_lens, int max_len, void* o, int B, int Hq, int Hkv,
                          int head_dim, double rope_theta, int w_pretrained, int w_local,
                          int remote_map, void* workspace, size_t workspace_bytes, void* stream);

/*
 * jl_bifocal_decode on a paged cache: keys and values live in pools of
 * fixed-size pages and each sequence lists its pages in a block table.
 *   k_pages, v_pages bf16 [n_pages, page_size, Hkv, head_dim] raw pools
 *   block_table      int32 [B, max_pages] DEVICE array: key k of sequence b
 *                    is row k % page_size of page block_table[b][k / page_size]
 *   kv_lens          int32 [B] DEVICE array, 1 <= kv_lens[b] <= max_pages * page_size
 *                    (clamped into that range as in jl_bifocal_decode)
 * page_size is a power of two, at least 16 (a 16-key step of the kernel never
 * straddles two pages).  Page indices outside [0, n_pages) are clamped into
 * the pool, so a bad table gives wrong values, never an out-of-bounds read.
 * Workspace as for jl_bifocal_decode with max_len = max_pages * page_size.
 * Other arguments, requirements and errors as in jl_bifocal_decode.
 */
int jl_bifocal_decode_paged(const void* q, const void* k_pages, const void* v_pages,
                            const int32_t* block_table, int max_pages, int page_size, int n_pages,
                            const int32_t* kv_lens, void* o, int B, int Hq, int Hkv,
                            int head_dim, double rope_theta, int w_pretrained, int w_local,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * jl_bifocal_decode_paged with a choice of remote map, as jl_bifocal_decode_map
 * offers it for dense caches: remote_map JL_REMOTE_ALIAS is
 * jl_bifocal_decode_paged bit for bit, JL_REMOTE_FREQ the Sec. 4.5 frequency
 * map with each sequence's factor from its own kv_len.  The workspace must
 * hold jl_decode_map_workspace_bytes(B, Hq, Hkv, max_pages * page_size,
 * head_dim, remote_map) bytes.  Other arguments and errors as in
 * jl_bifocal_decode_paged; remote_map outside {0, 1} -> JL_ERR_INVALID_ARG.
 */
int jl_bifocal_decode_paged_map(const void* q, const void* k_pages, const void* v_pages,
                                const int32_t* block_table, int max_pages, int page_size,
                                int n_pages, const int32_t* kv_lens, void* o, int B, int Hq,
                                int Hkv, int head_dim, double rope_theta, int w_pretrained,
                                int w_local, int remote_map, void* workspace,
                                size_t workspace_bytes, void* stream);

/* The vanilla counterpart of jl_bifocal_decode_paged. */
int jl_rope_attention_decode_paged(const void* q, const void* k_pages, const void* v_pages,
                                   const int32_t* block_table, int max_pages, int page_size,
                                   int n_pages, const int32_t* kv_lens, void* o, int B, int Hq,
                                   int Hkv, int head_dim, double rope_theta, void* workspace,
                                   size_t workspace_bytes, void* stream);

/*
 * Debug view of the schedule as the device computes it (Eqs. (2), (3), (5)),
 * for bit-exact tests.  All pointers are device pointers.
 *   lengths    int32 [n_lengths]              sequence lengths L (>= 1)
 *   positions  int32 [n_positions]            positions x (>= 0)
 *   group_out  int32 [n_lengths]              G(L)
 *   remote_out int32 [n_lengths, n_positions] f(x) = floor(x / G(L))
 *   offset_out int32 [n_lengths, n_positions] Delta(x) = f(x) - x
 */
int jl_debug_schedule(const int32_t* lengths, int n_lengths, const int32_t* positions,
                      int n_positions, int w_pretrained, int32_t* group_out, int32_t* remote_out,
                      int32_t* offset_out, void* stream);

/* Tile classes written by jl_debug_prefill_tiles. */
enum { JL_TILE_SKIP = 0, JL_TILE_LOCAL = 1, JL_TILE_REMOTE = 2, JL_TILE_MIXED = 3 };

/*
 * Debug view of the prefill kernel's tile classification (Eq. (1)'s window
 * boundary at tile granularity), computed on the device with the kernel's own
 * block sizes.  Writes int8 classes_out[n_qblocks, n_ktiles] (device) and the
 * block geometry to the host ints *block_q, *block_k, *n_qblocks, *n_ktiles.
 * classes_len is the capacity of classes_out in elements.
 */
int jl_debug_prefill_tiles(int L, int Hq, int Hkv, int w_local, int8_t* classes_out,
                           int64_t classes_len, int* block_q, int* block_k, int* n_qblocks,
                           int* n_ktiles, void* stream);

/*
 * Debug knob for tests, process-wide: the prefill kernels move a row's softmax
 * reference (and rescale the running output) when a key tile's largest score
 * in that row exceeds the reference by more than log2_bound (scores in log2
 * units), or lies more than log2_bound below it before anything was
 * accumulated; the default is 64, far from anything ordinary data reaches.
 * The fused and vanilla calls first run a pass without that check, which only
 * notes whether a tile's probability sum exceeded 2^log2_bound or a row's
 * total fell below 2^-log2_bound; such blocks are then rerun with the check.
 * A small bound (e.g. 3) sends almost every block through the rerun and the
 * rescale path, which tests use to check both.  Values outside [1, 100] leave
 * the setting unchanged.  Returns the previous value.  Not for use while
 * prefill calls are in flight.
 */
double jl_debug_prefill_rescale_log2(double log2_bound);

/*
 * Timing hook for benchmarks, process-wide.  which = 0: every later prefill
 * call that runs the fused or vanilla attention kernel (every prefill entry
 * point but the literal one's three window passes) records the HIP event
 * `start` on its stream right before that kernel and `stop` right after its
 * checked rerun, so hipEventElapsedTime(start, stop) is the attention alone
 * (the value-transpose kernel in front of it stays outside).  which = 1: the
 * same around the split kernel of every decode call that takes a workspace
 * (all but jl_bifocal_decode_noalloc; the reduce stays outside).
 * start, stop: hipEvent_t created and owned by the caller; NULL, NULL clears
 * the hook.  JL_ERR_INVALID_ARG for another `which` or when only one event is
 * NULL.  The events must outlive every call that records them.
 */
int jl_debug_kernel_events(int which, void* start, void* stop);

/* Frees the library-owned cos/sin tables and prefill scratch buffers on every
 * device (they are rebuilt on demand); waits for the streams that own scratch.
 * Must not race with running calls. */
void jl_release_caches(void);

#ifdef __cplusplus
}
#endif

#endif /* JETLONG_H */
