/*
 * vpp_chunk_attn.h -- chunked-prefill causal attention for AMD MI355X (gfx950).
 *
 * The operation (paper: "VPP: Virtual Pipeline Parallelism for Efficient
 * Chunked Prefill in Long-Context LLM Inference"):
 *
 *   Eq. (1), section 2.1: out = softmax(Q K^T * scale) V, causal: a token sees
 *   itself and the tokens before it.
 *   Section 2.4: in chunked prefill a prompt is cut into fixed-size chunks; the
 *   queries of a chunk attend to the cached prefix KV of all earlier chunks plus
 *   the earlier tokens of their own chunk, so a later chunk does more work. That
 *   growth (sections 1 and 5.1) is the cost curve that VPP's V-shaped stage
 *   layout balances.
 *
 * One call processes one chunk of query tokens. A chunk is a list of segments;
 * each segment is a run of consecutive tokens of one request (section 5.3 packs
 * the leading chunks of the next request behind the tail of the current one, so
 * a fixed-size chunk may hold several requests). Segment s holds chunk rows
 * cu_q[s] .. cu_q[s+1]-1; its row r has in-request position
 *     i = prefix_len[s] + (r - cu_q[s])
 * and sees the cache rows kv_start[s] + j for j = 0 .. i, and nothing of other
 * requests.
 *
 * Data types and layouts (all device memory, owned by the caller):
 *   q        bf16 [tokens][Hq][dqk]      strides q_stride_tok, q_stride_head
 *   k_cache  bf16 [rows][Hkv][dqk]       strides k_stride_tok, k_stride_head
 *   v_cache  bf16 [rows][Hkv][dv]        strides v_stride_tok, v_stride_head
 *   out      bf16 [tokens][Hq][dv]       strides o_stride_tok, o_stride_head
 *   lse      fp32 [Hq][...]              element h*lse_stride_head + r is chunk
 *                                        row r, head h (nullable)
 * Strides are in elements; the last dimension is contiguous; base pointers and
 * the token/head strides are multiples of 8 elements (16 bytes). Strides are
 * below 2^25 elements, and the cache row strides (k_stride_tok, v_stride_tok,
 * and kr_stride_tok of the split key layout) below 2^24: one 64-row key tile
 * must span less than 2^31 bytes. Larger strides are VPP_ERR_INVALID_ARG. Query head h
 * reads kv head h / (Hq / Hkv) (contiguous groups: grouped-query attention;
 * Hq == Hkv is multi-head attention, which is also how the MLA models of
 * section 6.1 are run in prefill, with dqk = 192 and dv = 128).
 * The chunk's own keys and values must already be in the cache (rows
 * kv_start[s] + prefix_len[s] .. kv_start[s] + prefix_len[s] + len - 1).
 *
 * Arithmetic: scores and the softmax in fp32, P rounded to bf16 for the P.V
 * product, fp32 accumulation; out rounded to bf16 (nearest even); lse is the
 * natural log of the softmax denominator of the scaled scores, fp32.
 *
 * Errors: every entry point returns a status and never aborts; a failed call
 * leaves its outputs unspecified and the plan usable.
 */
#ifndef VPP_CHUNK_ATTN_H
#define VPP_CHUNK_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    VPP_OK = 0,
    VPP_ERR_INVALID_ARG = 1, /* null/misaligned pointer, bad size or metadata */
    VPP_ERR_UNSUPPORTED = 2, /* head dims or options this build has no kernel for */
    VPP_ERR_WORKSPACE = 3,   /* workspace missing or smaller than the plan needs */
    VPP_ERR_HIP = 4,         /* a HIP runtime call or kernel launch failed */
    VPP_ERR_NOMEM = 5        /* host allocation failed */
} vpp_status_t;

/* Problem description, passed by value into a plan (copied). */
typedef struct {
    int32_t num_q_heads;      /* Hq > 0                                          */
    int32_t num_kv_heads;     /* Hkv > 0, Hq % Hkv == 0                          */
    int32_t head_dim_qk;      /* dqk                                             */
    int32_t head_dim_v;       /* dv; (dqk, dv) in {(64,64), (128,128), (192,128)} */
    float softmax_scale;      /* 0 => 1/sqrt(dqk)                                */
    int32_t causal;           /* must be 1: the causal rule of section 2.1       */
    int32_t max_chunk_tokens; /* bound on cu_q[n] over the plan's lifetime        */
    int32_t max_segments;     /* bound on the number of segments                  */
    int64_t max_kv_len;       /* bound on kv_start + prefix_len + len (cache rows) */
    int32_t num_splits;       /* split of the key range with an lse merge:
                                 -1 automatic, 1 off, 2..16 fixed                  */
} vpp_chunk_attn_config_t;

typedef struct vpp_chunk_attn_plan_s* vpp_chunk_attn_plan_t;

/*
 * Plan one chunk (host only; no device work, no GPU needed).
 *
 * Checks the segment metadata (host arrays: cu_q[n+1] with cu_q[0] = 0 and
 * non-decreasing; kv_start[n] >= 0; prefix_len[n] >= 0; every segment within
 * max_kv_len and the chunk within max_chunk_tokens; zero-length segments are
 * allowed and skipped), cuts the segments into query tiles, chooses the split
 * count, orders the work longest first and sizes the device workspace.
 *
 * *inout_plan == NULL creates a plan (owned by the library until
 * vpp_chunk_attn_destroy); a non-NULL plan is refilled in place with the same
 * config (cfg may be NULL then). Refilling never blocks: each run copies the
 * work list to the device from a pinned staging slot of its own (a ring of 4
 * per plan), and only a run that reuses a slot whose earlier copy is still in
 * flight waits, on the host, for that copy.
 * *workspace_bytes receives the bytes of device workspace vpp_chunk_attn_run
 * needs for this plan (always > 0). The arrays are not retained.
 */
vpp_status_t vpp_chunk_attn_plan(const vpp_chunk_attn_config_t* cfg,
                                 int32_t num_segments, const int32_t* cu_q,
                                 const int64_t* kv_start, const int64_t* prefix_len,
                                 vpp_chunk_attn_plan_t* inout_plan,
                                 size_t* workspace_bytes);

/*
 * Run a planned chunk, asynchronously on `stream` (a hipStream_t; NULL is the
 * default stream). Enqueues, in order: the copy of the plan's work list into
 * the workspace, the attention kernel, and -- when the plan splits the key
 * range -- the merge kernel. Never synchronizes the stream. All pointers are
 * caller-owned device memory that must stay valid until the stream reaches the
 * end of this work; lse may be NULL. The workspace (>= the planned bytes,
 * 256-byte aligned) must not be used by other work in flight.
 */
vpp_status_t vpp_chunk_attn_run(vpp_chunk_attn_plan_t plan,
                                const void* q, int64_t q_stride_tok, int64_t q_stride_head,
                                const void* k_cache, int64_t k_stride_tok, int64_t k_stride_head,
                                const void* v_cache, int64_t v_stride_tok, int64_t v_stride_head,
                                void* out, int64_t o_stride_tok, int64_t o_stride_head,
                                float* lse, int64_t lse_stride_head,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * Bytes of device scratch behind vpp_chunk_attn_run_noalloc: one static array
 * per GPU the library runs on, held until the process ends.
 */
#define VPP_NOALLOC_SCRATCH_BYTES (64u << 20)

/*
 * vpp_chunk_attn_run without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same plan, kernels, arguments and results
 * as vpp_chunk_attn_run: the same bits, split key ranges included. Its
 * workspace (the work list and, in split plans, the fp32 partials) is a static
 * device array of VPP_NOALLOC_SCRATCH_BYTES on the current device, whose
 * address the library looks up on its first call on that device. This call
 * makes no hipMalloc, hipFree, host-pinning or other allocating call: the work
 * list is copied to the device straight from the plan, whose host memory is
 * not pinned; HIP performs such a copy synchronously, so it is complete when
 * the call returns and the plan may be refilled at once. Nothing in the scratch
 * needs clearing between calls: every byte a run reads, the same run writes
 * first.
 * The array used is the current device's (hipGetDevice at the call): the
 * stream and every pointer must belong to that device. Calls on one GPU share
 * its array: calls whose work overlaps on that GPU (several streams, several
 * threads) race and give wrong results; serialize them.
 * Errors: VPP_ERR_WORKSPACE when the plan needs more than
 * VPP_NOALLOC_SCRATCH_BYTES (vpp_chunk_attn_plan's workspace size; large split
 * plans do), VPP_ERR_HIP when the array cannot be found on the current device,
 * and every error of vpp_chunk_attn_run.
 */
vpp_status_t vpp_chunk_attn_run_noalloc(vpp_chunk_attn_plan_t plan,
                                        const void* q, int64_t q_stride_tok, int64_t q_stride_head,
                                        const void* k_cache, int64_t k_stride_tok, int64_t k_stride_head,
                                        const void* v_cache, int64_t v_stride_tok, int64_t v_stride_head,
                                        void* out, int64_t o_stride_tok, int64_t o_stride_head,
                                        float* lse, int64_t lse_stride_head, void* stream);

/*
 * Split key layout of the MLA models the paper evaluates (section 6.1: its
 * DeepSeek model runs MLA attention, MHA-style in prefill): each key is the
 * concatenation of a per-head part and a part shared by all heads,
 *   K[j][h] = ( k_nope[j][h][0..127], k_rope[j][0..63] ),   dqk = 192, dv = 128,
 * so the shared 64 dims are stored once per row instead of once per head (a
 * third less key memory and traffic). Layouts (device memory, caller-owned):
 *   k_nope bf16 [rows][Hkv][128]  strides kn_stride_tok, kn_stride_head
 *   k_rope bf16 [rows][64]        stride kr_stride_tok
 * Everything else (q with dqk = 192, v, out, lse, plan, workspace, stream) is
 * as for vpp_chunk_attn_run, and so are the results: the same bits as
 * vpp_chunk_attn_run over the concatenated keys, split key ranges included.
 * Errors: VPP_ERR_UNSUPPORTED unless the plan's head dims are (192, 128);
 * VPP_ERR_INVALID_ARG for a null or misaligned k_rope or a bad kr_stride_tok
 * (>= 64, a multiple of 8); every error of vpp_chunk_attn_run.
 */
vpp_status_t vpp_chunk_attn_run_mla(vpp_chunk_attn_plan_t plan,
                                    const void* q, int64_t q_stride_tok, int64_t q_stride_head,
                                    const void* k_nope, int64_t kn_stride_tok, int64_t kn_stride_head,
                                    const void* k_rope, int64_t kr_stride_tok,
                                    const void* v_cache, int64_t v_stride_tok, int64_t v_stride_head,
                                    void* out, int64_t o_stride_tok, int64_t o_stride_head,
                                    float* lse, int64_t lse_stride_head,
                                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * Paged KV cache. The paper's system runs inside a serving engine (vLLM,
 * sections 5.4 and 6.1) whose KV cache is cut into fixed-size pages assigned
 * to requests through block tables; the chunk semantics are unchanged
 * (section 2.4). Layout (device memory, caller-owned):
 *   k_pages  bf16 [num_pages][page_size][Hkv][dqk]  strides k_stride_page,
 *                                                   k_stride_tok, k_stride_head
 *   v_pages  bf16 [num_pages][page_size][Hkv][dv]   likewise
 *   block_table int32, row s (segment s of the plan) at block_table +
 *            s * block_table_stride: entry i is the page holding cache rows
 *            i*page_size .. (i+1)*page_size - 1 of that segment's request.
 * The plan's kv_start[s] is the cache row of in-request position 0 (normally
 * 0) and must be a multiple of 64; cache row j of segment s is row
 * j % page_size of page block_table[s][j / page_size]. page_size is a power of
 * two >= 64 (a 64-key tile never straddles a page). The table must cover every
 * row the chunk reads (kv_start + prefix_len + len rows per segment). Page
 * indices are clamped to [0, num_pages - 1] on the device, so a bad entry gives
 * wrong values, never an out-of-range read. Arithmetic, outputs, workspace and
 * stream semantics are those of vpp_chunk_attn_run, and so are the results:
 * the same bits as a contiguous cache holding the same rows.
 * Errors: VPP_ERR_INVALID_ARG for a bad page size, page stride, block table
 * pointer or kv_start alignment, plus every error of vpp_chunk_attn_run.
 */
vpp_status_t vpp_chunk_attn_run_paged(vpp_chunk_attn_plan_t plan,
                                      const void* q, int64_t q_stride_tok, int64_t q_stride_head,
                                      const void* k_pages, int64_t k_stride_page, int64_t k_stride_tok,
                                      int64_t k_stride_head,
                                      const void* v_pages, int64_t v_stride_page, int64_t v_stride_tok,
                                      int64_t v_stride_head,
                                      int32_t page_size, int32_t num_pages,
                                      const int32_t* block_table, int64_t block_table_stride,
                                      void* out, int64_t o_stride_tok, int64_t o_stride_head,
                                      float* lse, int64_t lse_stride_head,
                                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * Write a chunk's new keys and values into a paged cache (asynchronously on
 * `stream`): token t's rows k_new[t] [Hkv][dqk] and v_new[t] [Hkv][dv] go to
 * slot slot_mapping[t] = page * page_size + row of k_pages / v_pages (layouts
 * as for vpp_chunk_attn_run_paged). Slots outside [0, num_pages * page_size)
 * are skipped (e.g. -1 for padding). This is the cache write that must precede
 * the chunk's attention (section 2.4). Head dims are multiples of 8, at most
 * 1024; pointers 16-byte aligned (slot_mapping: 8-byte, int64 device array);
 * strides multiples of 8 elements. Two tokens mapped to one slot race.
 * Errors: VPP_ERR_INVALID_ARG, VPP_ERR_HIP (launch failure).
 */
vpp_status_t vpp_kv_append_paged(const void* k_new, int64_t kn_stride_tok, int64_t kn_stride_head,
                                 const void* v_new, int64_t vn_stride_tok, int64_t vn_stride_head,
                                 void* k_pages, int64_t k_stride_page, int64_t k_stride_tok,
                                 int64_t k_stride_head,
                                 void* v_pages, int64_t v_stride_page, int64_t v_stride_tok,
                                 int64_t v_stride_head,
                                 int32_t num_tokens, int32_t num_kv_heads, int32_t head_dim_qk,
                                 int32_t head_dim_v, int32_t page_size, int32_t num_pages,
                                 const int64_t* slot_mapping, void* stream);

/*
 * Host helper: the slot of each chunk row for vpp_kv_append_paged, from the
 * same segment metadata as vpp_chunk_attn_plan and a host copy of the block
 * table (rows of pages_per_row valid entries, block_table_stride apart):
 * slot_mapping[r] (host, cu_q[n] entries) = page * page_size + row of cache
 * row kv_start[s] + prefix_len[s] + (r - cu_q[s]). Errors: VPP_ERR_INVALID_ARG
 * for malformed metadata, a row past its table row, or a negative page.
 */
vpp_status_t vpp_paged_slot_mapping(int32_t num_segments, const int32_t* cu_q,
                                    const int64_t* kv_start, const int64_t* prefix_len,
                                    const int32_t* block_table, int64_t block_table_stride,
                                    int32_t pages_per_row, int32_t page_size,
                                    int64_t* slot_mapping);

/* Free a plan (NULL is ignored). Waits for the device to finish reading its
 * work list first. */
void vpp_chunk_attn_destroy(vpp_chunk_attn_plan_t plan);

/* Static text for a status value. */
const char* vpp_status_str(vpp_status_t status);

/* Summary of a plan, for callers that size buffers or report work. */
typedef struct {
    int32_t num_tiles;        /* query tiles (per head) in the chunk               */
    int32_t num_splits;       /* split count chosen (1 = no merge pass)            */
    int32_t num_work_items;   /* work-list entries: two per slot                   */
    int32_t block_m;          /* query rows per tile                               */
    int32_t block_n;          /* keys per inner step                               */
    int32_t num_tokens;       /* cu_q[n]                                           */
    int64_t workspace_bytes;  /* same value vpp_chunk_attn_plan returned           */
    double pairs;             /* visible (query, key) pairs per head               */
    int32_t num_slots;        /* work slots = workgroups per head of the launch    */
} vpp_chunk_attn_plan_info_t;

vpp_status_t vpp_chunk_attn_plan_info(vpp_chunk_attn_plan_t plan,
                                      vpp_chunk_attn_plan_info_t* info);

/* One planned work item, as the kernel reads it (rows and keys in
 * in-request coordinates). */
typedef struct {
    int32_t row0;      /* first chunk row of the tile                         */
    int32_t nrows;     /* rows in the tile (1 .. block_m)                      */
    int32_t pos0;      /* in-request position of row0                          */
    int32_t key_begin; /* keys [key_begin, key_end) of the request             */
    int32_t key_end;
    int32_t split;     /* split index, 0 .. num_splits-1                       */
    int64_t kv_base;   /* cache row of the request's position 0                */
} vpp_chunk_attn_work_item_t;

/* Copy up to `capacity` work items of the plan, in launch order; *count gets
 * the plan's item count. Entries 2m and 2m+1 form work slot m, which one
 * workgroup per head runs: the first entry's tile with its keys ascending, then
 * the second's (the partner tile from the other end of the same segment, in the
 * same split piece) with its keys descending. A second entry with nrows = 0 is
 * empty. Every (tile, split piece) appears exactly once. */
vpp_status_t vpp_chunk_attn_plan_items(vpp_chunk_attn_plan_t plan,
                                       vpp_chunk_attn_work_item_t* items,
                                       int32_t capacity, int32_t* count);

#ifdef __cplusplus
}
#endif
#endif /* VPP_CHUNK_ATTN_H */
