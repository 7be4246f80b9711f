/*
 * pcr.h -- C ABI of libpcr: the per-layer prefix-reuse prefill step on MI355X (gfx950).
 *
 * The operation (PCR, Sec. 2.2, 4.3 and 5; Alg. 1): a request's tokens split
 * into a cached prefix of p tokens, whose K/V already exist in pinned host
 * memory, and an uncached suffix of s tokens. For every layer, the prefix K/V
 * blocks are copied into a paged GPU KV pool (Sec. 5: fixed 16-token blocks
 * mapped through a per-sequence block table, one pool per layer), the
 * suffix's new K/V rows are written into the pool, and causal attention runs
 * for the s suffix rows over all p + s keys. With exact prefix matching the
 * result equals full prefill's output for those rows (Sec. 2.2). A two-stream
 * pipeline overlaps layer l's compute with the loads of later layers
 * (Sec. 4.3: only about one layer's load stays exposed when per-layer compute
 * exceeds per-layer load).
 *
 * Conventions for every entry point:
 *   - Ownership: the caller owns every buffer. Device buffers are plain
 *     device pointers (e.g. from hipMalloc or a framework allocator); host
 *     KV stores must be pinned (hipHostMalloc). The library keeps no pointer
 *     after a call returns.
 *   - Asynchrony: calls that take a stream only enqueue work on it and do
 *     not synchronise (pcr_pipeline_run with timing output is the one
 *     exception). Inputs must stay alive until the stream has passed the work.
 *   - Streams are hipStream_t values passed as void*; NULL is the default stream.
 *   - Errors: argument checks run on the host before anything is enqueued and
 *     return a negative pcr_status; pcr_last_error() then holds a message
 *     (per thread). Faults inside kernels surface at the caller's next
 *     synchronisation. No C++ exception crosses this interface.
 *   - Supported shapes: bf16 K/V/Q, block_size 16, head_dim 64 or 128,
 *     num_q_heads a multiple of num_kv_heads. Anything else returns
 *     PCR_ERR_UNSUPPORTED.
 *   - Empty work (n = 0 pairs, T = 0 tokens, a sequence with s = 0) is a no-op
 *     returning PCR_OK.
 *
 * KV block layout (one layer; K and V are separate arrays of num_blocks blocks;
 * each block holds num_kv_heads payloads of block_size * head_dim bf16):
 *   K of (block blk, kv head g, slot o, dim x) at ((blk*Hkv + g)*bs + o)*d + x
 *   V of (block blk, kv head g, slot o, dim x) at ((blk*Hkv + g)*d + x)*bs + o
 * Host stores use the same per-block layout, so a load is a bitwise block copy.
 * Logical token t of sequence b is slot t % bs of pool block block_tables[b][t / bs].
 * Query head h attends with kv head h / (num_q_heads / num_kv_heads).
 */
#ifndef PCR_H_
#define PCR_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum pcr_status {
    PCR_OK = 0,
    PCR_ERR_INVALID_ARG = -1,  /* null pointer, bad size, id out of range, inconsistent shapes */
    PCR_ERR_UNSUPPORTED = -2,  /* valid but unsupported shape (head_dim, block_size, ...) */
    PCR_ERR_NOT_PINNED = -3,   /* a host KV store is not pinned, device-accessible memory */
    PCR_ERR_HIP = -4           /* a HIP runtime call failed while enqueuing */
} pcr_status;

/* One layer's paged KV pool in device memory. */
typedef struct pcr_kv_pool {
    void *k;
    void *v;
    int32_t num_blocks;
    int32_t block_size;
    int32_t num_kv_heads;
    int32_t head_dim;
} pcr_kv_pool;

/* One layer's host KV store (pinned host memory, same per-block layout). */
typedef struct pcr_host_kv {
    const void *k;
    const void *v;
    int64_t num_blocks;
    int32_t block_size;
    int32_t num_kv_heads;
    int32_t head_dim;
} pcr_host_kv;

/* How pcr_load_kv_layer moves blocks over the host link. */
typedef enum pcr_load_method {
    PCR_LOAD_AUTO = 0,          /* the library's default (the measured fastest) */
    PCR_LOAD_DMA_BATCH = 1,     /* one hipMemcpyBatchAsync per call; runs of consecutive
                                   blocks merged into one copy */
    PCR_LOAD_DMA_PER_BLOCK = 2, /* one hipMemcpyAsync per block and per K/V (the
                                   block-by-block baseline of Sec. 5) */
    PCR_LOAD_KERNEL_PULL = 3,   /* a copy kernel on the given stream reads the pinned host
                                   pages directly and writes the pool blocks */
    PCR_LOAD_DMA_STAGED = 4     /* through a device workspace: the copy engines move whole
                                   runs of consecutive host blocks over the host link and a
                                   kernel scatters (load) or gathers (offload) the pool blocks
                                   at HBM speed; only with the *_staged entry points */
} pcr_load_method;

/*
 * pcr_plan -- host-side planning of one batch (Alg. 1, planning loop:
 * each cached block of a scheduled request goes on the host-to-GPU list;
 * only the unmatched tokens are computed).
 *
 * In (host arrays):
 *   prefix_lens[B], suffix_lens[B]        cached and new token counts (>= 0)
 *   block_tables[B][max_blocks]           pool block of every logical block; entries
 *                                         past ceil((p+s)/bs) are ignored
 *   host_blocks[B][max_host_blocks]       host-store block of every logical prefix
 *                                         block; entries past ceil(p/bs) are ignored
 * Out (host arrays, caller-allocated):
 *   src_blocks[cap_pairs], dst_blocks[cap_pairs], *n_pairs
 *       the load list, sequence by sequence, logical block ascending; a pair equal
 *       to an earlier one (a prefix block shared between sequences) is listed once.
 *       cap_pairs = sum_b ceil(p_b / bs) always suffices.
 *   slot_mapping[sum_b s_b]   pool slot (block*bs + offset) of each new token,
 *                             sequences in order
 *   cu_suffix[B+1]            prefix sums of suffix_lens
 * Errors (PCR_ERR_INVALID_ARG): a needed block id < 0; a pool block named as the
 * destination of two different host blocks; a new token's slot already taken, or
 * inside a pool block another sequence loads; capacity too small.
 * Touches no GPU.
 */
pcr_status pcr_plan(int32_t B, const int32_t *prefix_lens, const int32_t *suffix_lens,
                    const int32_t *block_tables, int32_t max_blocks,
                    const int32_t *host_blocks, int32_t max_host_blocks, int32_t block_size,
                    int32_t *src_blocks, int32_t *dst_blocks, int32_t cap_pairs, int32_t *n_pairs,
                    int32_t *slot_mapping, int32_t *cu_suffix);

/*
 * pcr_load_kv_layer -- enqueue the host-to-pool copy of one layer's cached blocks
 * (Sec. 5: one chunk's blocks land in non-consecutive pool blocks; Alg. 1
 * "LayerwiseUpload"). For each i < n: pool block dst_blocks[i] of dst (K and V,
 * all kv heads) becomes a bitwise copy of host block src_blocks[i] of src.
 * src_blocks / dst_blocks are host arrays, range-checked on the host; dst ids
 * must be distinct. src must be pinned (PCR_ERR_NOT_PINNED otherwise). Shapes of
 * src and dst must match. The caller records an event on copy_stream after the
 * call to order later compute behind the copy.
 */
pcr_status pcr_load_kv_layer(const pcr_host_kv *src, const int32_t *src_blocks,
                             const pcr_kv_pool *dst, const int32_t *dst_blocks, int32_t n,
                             void *copy_stream);

/* The same, with the copy method chosen by the caller. */
pcr_status pcr_load_kv_layer_method(const pcr_host_kv *src, const int32_t *src_blocks,
                                    const pcr_kv_pool *dst, const int32_t *dst_blocks, int32_t n,
                                    pcr_load_method method, void *copy_stream);

/*
 * pcr_plan_offload -- the GPU-to-host list of one batch (Alg. 1: a chunk of a
 * scheduled request that no cache tier holds is computed, then goes on the
 * GPU-to-CPU list, "LayerwiseDownload"). For each sequence b, every whole chunk of
 * chunk_tokens tokens (aligned to multiples of chunk_tokens from the sequence
 * start) that lies entirely inside the computed range [prefix_lens[b],
 * prefix_lens[b] + suffix_lens[b]) is listed block by block, sequences in order:
 * src_blocks[i] is its pool block (from block_tables) and dst_blocks[i] =
 * first_dst_block + i (host-store blocks in consecutive order, ready to become the
 * chunks' cache entries). A trailing partial chunk is not offloaded.
 *   chunk_tokens   a positive multiple of block_size
 *   cap            capacity of src_blocks / dst_blocks; *n_pairs receives the count
 * Errors: PCR_ERR_INVALID_ARG for negative lengths, a chunk size that is not a
 * multiple of the block size, a missing pool block (-1 or past max_blocks), or
 * more pairs than cap (nothing useful is written then).
 */
pcr_status pcr_plan_offload(int32_t B, const int32_t *prefix_lens, const int32_t *suffix_lens,
                            const int32_t *block_tables, int32_t max_blocks, int32_t block_size,
                            int32_t chunk_tokens, int32_t first_dst_block,
                            int32_t *src_blocks, int32_t *dst_blocks, int32_t cap, int32_t *n_pairs);

/*
 * pcr_offload_kv_layer -- enqueue the pool-to-host copy of one layer's new blocks
 * (Alg. 1 "LayerwiseDownload"; Sec. 4.3: offloading a layer starts as soon as
 * that layer's computation ends; Sec. 5: on a stream of its own). For each i < n:
 * host block dst_blocks[i] of dst becomes a bitwise copy of pool block
 * src_blocks[i] of src (K and V, all kv heads). Host arrays, range-checked on the
 * host; dst ids must be distinct; dst must be pinned (PCR_ERR_NOT_PINNED
 * otherwise). The caller orders the call after the compute that wrote the
 * blocks (an event from the compute stream).
 * Methods: PCR_LOAD_AUTO and PCR_LOAD_KERNEL_PULL select the copy kernel, which
 * here reads the pool and writes the pinned host pages directly;
 * PCR_LOAD_DMA_PER_BLOCK issues one hipMemcpyAsync per block and per K/V;
 * PCR_LOAD_DMA_BATCH one batched copy (PCR_ERR_UNSUPPORTED without it).
 */
pcr_status pcr_offload_kv_layer(const pcr_kv_pool *src, const int32_t *src_blocks,
                                const pcr_host_kv *dst, const int32_t *dst_blocks, int32_t n,
                                void *stream);
pcr_status pcr_offload_kv_layer_method(const pcr_kv_pool *src, const int32_t *src_blocks,
                                       const pcr_host_kv *dst, const int32_t *dst_blocks, int32_t n,
                                       pcr_load_method method, void *stream);

/*
 * The staged forms of the two copies (PCR_LOAD_DMA_STAGED). workspace: device
 * memory owned by the caller, 16-byte aligned, at least 2 * n * block bytes
 * (block bytes = block_size * num_kv_heads * head_dim * 2); its contents are
 * scratch. Work on one stream is ordered, so one workspace serves every call on
 * that stream; calls on different streams that may overlap need their own.
 * Offload: a kernel gathers the listed pool blocks into the workspace, then one
 * copy-engine transfer per run of consecutive dst host blocks. Load: one transfer
 * per run of consecutive src host blocks into the workspace, then a kernel
 * scatters the blocks into the pool. The long host-link transfers then occupy no
 * compute unit (a kernel that writes host memory directly slows kernels running
 * beside it far more than the copy engines do). PCR_ERR_INVALID_ARG if the
 * workspace is missing or too small.
 */
pcr_status pcr_offload_kv_layer_staged(const pcr_kv_pool *src, const int32_t *src_blocks,
                                       const pcr_host_kv *dst, const int32_t *dst_blocks, int32_t n,
                                       void *workspace, int64_t workspace_bytes, void *stream);
pcr_status pcr_load_kv_layer_staged(const pcr_host_kv *src, const int32_t *src_blocks,
                                    const pcr_kv_pool *dst, const int32_t *dst_blocks, int32_t n,
                                    void *workspace, int64_t workspace_bytes, void *stream);

/*
 * pcr_append_kv -- write the new tokens' K/V into the pool (the KV write that
 * computing the uncached tokens implies, Sec. 4.3).
 *   k_new, v_new   device, bf16 [T][Hkv][d] (row-major, contiguous)
 *   slot_mapping   device, int32 [T]: pool slot of token t (block*bs + offset);
 *                  slots must be distinct; a token whose slot is negative or
 *                  outside the pool is skipped by the kernel (no error is
 *                  reported: the values live in device memory)
 * When a prefix ends inside a block, that block must be loaded before this call
 * (the load copies the whole block; the append then fills its free slots).
 */
pcr_status pcr_append_kv(const pcr_kv_pool *pool, const void *k_new, const void *v_new,
                         const int32_t *slot_mapping, int32_t T, void *stream);

/*
 * pcr_prefix_prefill_attn -- causal GQA attention of the suffix rows over the
 * cached prefix plus the suffix, read through the block table (Sec. 2.2, 5).
 * For sequence b, query head h, suffix row i (absolute position p_b + i), and
 * keys j in [0, p_b + i]:  out = sum_j softmax_j(sm_scale * <q, k_j>) v_j.
 *   q              device bf16 [T][Hq][d]; T = cu_suffix[B]
 *   block_tables   device int32 [B][max_blocks]
 *   prefix_lens    device int32 [B];  cu_suffix device int32 [B+1]
 *   host_prefix_lens, host_cu_suffix   host copies of the same; they must equal the
 *                  device arrays. The launch takes the lengths from these (they size it
 *                  and travel in its arguments); the device arrays must be valid
 *                  (non-NULL) but are not read.
 *   out            device bf16 [T][Hq][d]; fp32 accumulation, rounded to nearest even
 *   sm_scale       finite and > 0 (else PCR_ERR_INVALID_ARG)
 * Numerics: scores <q, k_j> and their scaling are fp32; the probabilities enter the
 * product with V rounded to bf16 and each row is normalised by the sum of those
 * rounded values, so the weights sum to one for any softmax sharpness. Per output
 * element the error is about 2^-8 max_j |v_j - out| plus half a bf16 ulp of out.
 * Every key position j <= p_b + s_b - 1 must hold valid data (loaded or appended);
 * slots past p_b + s_b are never read into the result.
 * Mixed batches: a sequence with s_b = 1 (a decode row) and Hq / Hkv <= 16 is
 * computed in the same launch by a decode workgroup (the key range split over its
 * waves, the same numerics as pcr_decode_attn), and such rows are spread over the
 * prefill row tiles of the launch so that they run beside them.
 */
pcr_status pcr_prefix_prefill_attn(const void *q, const pcr_kv_pool *pool,
                                   const int32_t *block_tables, int32_t max_blocks,
                                   const int32_t *prefix_lens, const int32_t *cu_suffix,
                                   const int32_t *host_prefix_lens, const int32_t *host_cu_suffix,
                                   int32_t B, int32_t num_q_heads, float sm_scale, void *out,
                                   void *stream);

/*
 * pcr_prefill_attn_set_schedule -- how pcr_prefix_prefill_attn (and the pipelines'
 * attention) divides a launch among workgroups; a tuning and testing control, not
 * part of the method. Every schedule computes the same result (Sec. 2.2).
 *   PCR_ATTN_SCHEDULE_AUTO (the default): row halves when that still gives at
 *     least two workgroups per compute unit, else key halves; pcr_pipeline_run and
 *     pcr_pipeline_run_offload, whose pull-kernel loads share the compute units
 *     with the attention, take key halves (shorter workgroups let the copy
 *     workgroups onto a compute unit sooner);
 *   PCR_ATTN_SCHEDULE_KEY_HALVES: 128 packed query rows per workgroup, the two
 *     wave groups on the two halves of the key range, merged at the end;
 *   PCR_ATTN_SCHEDULE_ROW_HALVES: 256 packed query rows per workgroup, each wave
 *     group on 128 of them over the whole key range, both reading one copy of
 *     each K/V tile (half the workgroups, each with one start-up and no merge for
 *     twice the work, and half the tile loads per row).
 * A batch with more than 128 sequences with new tokens runs as consecutive launches
 * on the stream, the sequences (longest context first) dealt round robin so that
 * every launch gets the same mix; the schedule is chosen per launch.
 * Process-wide; takes effect at the next launch. PCR_ERR_INVALID_ARG for an
 * unknown value.
 */
#define PCR_ATTN_SCHEDULE_AUTO 0
#define PCR_ATTN_SCHEDULE_KEY_HALVES 1
#define PCR_ATTN_SCHEDULE_ROW_HALVES 2
pcr_status pcr_prefill_attn_set_schedule(int32_t schedule);

/*
 * pcr_decode_attn -- one decode step: attention of one new query token per
 * sequence over every key of that sequence (Sec. 2.2 with a one-token suffix:
 * the output equals the last row of a full prefill of the sequence).
 * For sequence b, query head h and keys j in [0, n_b):
 *     out = sum_j softmax_j(sm_scale * <q, k_j>) v_j
 * where n_b = context_lens[b] counts the cached tokens plus the token being
 * decoded, whose K/V must already be in the pool (pcr_append_kv).
 *   q                  device bf16 [B][Hq][d], 16-byte aligned
 *   block_tables       device int32 [B][max_blocks]; entries past ceil(n_b/bs) are not read
 *   context_lens       device int32 [B]; host_context_lens: host copy of the same
 *                      (sizes the launch; the two must be equal)
 *   out                device bf16 [B][Hq][d], 16-byte aligned; fp32 accumulation,
 *                      rounded to nearest even
 *   workspace          device memory owned by the caller, 16-byte aligned, of
 *                      pcr_decode_attn_workspace_size(B, Hq, Hkv, d, max_b n_b) bytes
 *                      (NULL when that is 0); its contents are scratch. One workspace
 *                      serves every call ordered on one stream; calls that may overlap
 *                      need their own.
 * The key range of each (sequence, kv head) is split into chunks processed in
 * parallel and merged exactly (in LDS, or through the workspace and a second
 * kernel on the same stream), so the result does not depend on the split beyond
 * fp32 rounding. The chunk size follows the total count of keys when that gives
 * shorter chunks than the largest context alone (ragged batches: long sequences
 * get more chunks than short ones) and the workspace holds that plan; otherwise
 * it follows the largest context, which needs at most the workspace that
 * pcr_decode_attn_workspace_size reported before ragged plans existed (the error
 * message names the size needed). The plan depends only on the host context
 * lengths and the workspace size, so repeated calls give identical bits. Numerics as for
 * pcr_prefix_prefill_attn (fp32 scores, bf16 probabilities, rows normalised by
 * the rounded values); sm_scale must be finite and > 0.
 * Errors: PCR_ERR_UNSUPPORTED if Hq/Hkv > 16 (pcr_prefix_prefill_attn with
 * one-token suffixes covers that case); PCR_ERR_INVALID_ARG if some n_b < 1,
 * ceil(n_b/bs) > max_blocks, or the workspace is missing or too small (the
 * message names the size needed). B = 0 is a no-op.
 */
pcr_status pcr_decode_attn(const void *q, const pcr_kv_pool *pool, const int32_t *block_tables,
                           int32_t max_blocks, const int32_t *context_lens, const int32_t *host_context_lens,
                           int32_t B, int32_t num_q_heads, float sm_scale, void *out, void *workspace,
                           int64_t workspace_bytes, void *stream);

/*
 * pcr_decode_attn_noalloc -- pcr_decode_attn without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc). Same arguments, result and
 * numerics as pcr_decode_attn; the partial results of the chunk merge go to a
 * scratch array of PCR_DECODE_NOALLOC_SCRATCH_BYTES (16 MiB) that the library
 * holds per device until the process ends (its address is taken on the first call
 * on each device). The call allocates nothing and calls no allocating routine.
 * With a workspace of pcr_decode_attn_workspace_size bytes, pcr_decode_attn makes
 * the same plan as this entry point and gives the same bits.
 * Every call on one device shares that device's scratch, which keeps the last
 * call's contents (nothing needs clearing: each call writes every entry it reads
 * back), so calls on one device that may overlap (different streams, or host
 * threads without ordering) race; order them on one stream.
 * Errors: as pcr_decode_attn, and PCR_ERR_UNSUPPORTED when the batch would need
 * more scratch than the maximum (the plan by the largest context needs at most
 * about 11 MiB for any batch on a 256-compute-unit GPU, and the plan by total keys
 * is taken only when it fits); the message names both sizes.
 */
#define PCR_DECODE_NOALLOC_SCRATCH_BYTES (16 << 20)
pcr_status pcr_decode_attn_noalloc(const void *q, const pcr_kv_pool *pool, const int32_t *block_tables,
                                   int32_t max_blocks, const int32_t *context_lens,
                                   const int32_t *host_context_lens, int32_t B, int32_t num_q_heads,
                                   float sm_scale, void *out, void *stream);

/*
 * pcr_decode_attn_workspace_size -- bytes of workspace with which pcr_decode_attn
 * takes its best plan on the current device for any batch of B sequences whose
 * context lengths are at most max_context (0 when every such batch is handled
 * without one); never decreases as max_context grows, and never exceeds
 * PCR_DECODE_NOALLOC_SCRATCH_BYTES beyond what the plan by the largest context
 * needs. Queries the device's compute-unit count; PCR_ERR_HIP when no device is
 * usable.
 */
pcr_status pcr_decode_attn_workspace_size(int32_t B, int32_t num_q_heads, int32_t num_kv_heads,
                                          int32_t head_dim, int32_t max_context, int64_t *bytes);

/*
 * pcr_gather_kv -- read tokens back out of the pool in logical order (the
 * staging step of a layer-wise offload, Sec. 4.3; also a test aid).
 * For each sequence b, tokens starts[b] .. starts[b]+lens[b]-1 go to rows
 * cu_out[b] .. of k_out / v_out (device bf16 [total][Hkv][d]).
 *   block_tables device [B][max_blocks]; starts, lens, cu_out device int32
 *   total = host copy of cu_out[B] (sizes the launch)
 */
pcr_status pcr_gather_kv(const pcr_kv_pool *pool, const int32_t *block_tables, int32_t max_blocks,
                         const int32_t *starts, const int32_t *cu_out, int32_t B, int32_t total,
                         void *k_out, void *v_out, void *stream);

/* Per-layer device inputs and outputs for pcr_pipeline_run. */
typedef struct pcr_layer_io {
    pcr_host_kv host;     /* this layer's pinned host store */
    pcr_kv_pool pool;     /* this layer's pool */
    const void *q;        /* device bf16 [T][Hq][d] */
    const void *k_new;    /* device bf16 [T][Hkv][d] */
    const void *v_new;    /* device bf16 [T][Hkv][d] */
    void *out;            /* device bf16 [T][Hq][d] */
} pcr_layer_io;

/* The batch structure shared by every layer (from pcr_plan). */
typedef struct pcr_batch {
    const int32_t *src_blocks;        /* host [n_pairs] */
    const int32_t *dst_blocks;        /* host [n_pairs] */
    int32_t n_pairs;
    const int32_t *slot_mapping;      /* device [T] */
    int32_t T;
    const int32_t *block_tables;      /* device [B][max_blocks] */
    int32_t max_blocks;
    const int32_t *prefix_lens;       /* device [B] */
    const int32_t *cu_suffix;         /* device [B+1] */
    const int32_t *host_prefix_lens;  /* host [B] */
    const int32_t *host_cu_suffix;    /* host [B+1] */
    int32_t B;
    int32_t num_q_heads;
    float sm_scale;
} pcr_batch;

/*
 * pcr_pipeline_run -- the layer-wise overlapped step (Sec. 4.3; Alg. 1
 * "LayerwiseUpload" and "WaitForUploadEvents"). Every layer's load goes on
 * copy_stream, each followed by an event; compute_stream waits on layer l's
 * event, then runs layer l's append and attention. The host queues layer by
 * layer (load l, then compute l), so the copy stream runs the loads back to back
 * while the compute stream starts as soon as the first load is done. Layers are
 * independent here (each layer's Q and new K/V are inputs).
 * timing_ms: NULL, or host float[4*n_layers + 2]. When given, the call waits for
 * the last layer and fills, per layer l: [4l] load ms, [4l+1] compute ms
 * (append + attention), [4l+2] compute-stream wait before the layer (exposed
 * load), [4l+3] end of the layer's compute relative to the pipeline start; then
 * [4n] the whole pipeline ms and [4n+1] the sum of compute ms.
 * Overlap needs copy_stream and compute_stream on different hardware queues:
 * HIP maps a process's streams, in creation order, onto GPU_MAX_HW_QUEUES
 * hardware queues (4 unless the environment sets it), and two streams on one
 * queue run in series. Create these streams before others, or raise
 * GPU_MAX_HW_QUEUES before HIP starts (the same holds for the three streams of
 * pcr_pipeline_run_offload).
 * Every layer must have its own pool: nothing orders a later layer's load (copy
 * stream) after an earlier layer's attention (compute stream), so layers sharing
 * pool memory would race. Pool K/V base pointers repeated across layers (or a
 * layer's K equal to its V) are refused with PCR_ERR_INVALID_ARG; pools that
 * overlap at different base addresses are not detected and are the caller's error.
 * Errors: the pools' distinctness and the attention arguments of every layer
 * (batch-wide lengths, heads, sm_scale, block table size; each layer's pool, q
 * and out) are checked before anything is queued, and an error there leaves the
 * streams untouched. A later
 * error (a load's block list or unpinned host memory, found when that layer's
 * load is queued; a failed launch) returns with the earlier layers' work still
 * queued: it runs to completion, and the pools' contents are then unspecified.
 */
pcr_status pcr_pipeline_run(const pcr_layer_io *layers, int32_t n_layers, const pcr_batch *batch,
                            pcr_load_method method, void *copy_stream, void *compute_stream,
                            float *timing_ms);

/*
 * pcr_pipeline_run_staged -- pcr_pipeline_run with every layer's load staged
 * (Sec. 5: the layer's blocks go over the host link as batched copy-engine
 * transfers on their own stream). Layer l's host blocks batch->src_blocks are
 * moved by the copy engines into a workspace slot on copy_stream (one transfer
 * per run of consecutive host blocks, K then V), then a kernel on scatter_stream
 * writes them to pool blocks batch->dst_blocks; compute_stream waits for that
 * scatter, then runs layer l's append and attention. The transfers hold no
 * compute unit while attention runs beside them. workspace: device memory,
 * 16-byte aligned, of workspace_bytes >= one slot = 2 * n_pairs * block_size *
 * num_kv_heads * head_dim * 2 bytes (pcr_load_kv_layer_staged's workspace); it
 * holds floor(workspace_bytes / slot) slots (at most n_layers), layer l using
 * slot l mod slots, and the transfer into a slot waits for the scatter that last
 * read it: with two or more slots, layer l+1's transfer runs while layer l is
 * scattered. The workspace must not be used by other work until the pipeline has
 * run; the first transfers wait for the work already queued on scatter_stream
 * and compute_stream, and the first scatter for compute_stream. The three
 * streams must differ (and overlap only on different hardware queues, as for
 * pcr_pipeline_run). Every layer's pool must have the same block shape.
 * timing_ms and errors as pcr_pipeline_run; [4l] (load ms) spans the layer's
 * transfers and scatter. PCR_ERR_INVALID_ARG for a missing, misaligned or too
 * small workspace or equal streams, before anything is queued.
 * Choice of form: when a layer's compute takes at least as long as its load,
 * this form leaves the attention its whole device and exposes less of the loads
 * than pcr_pipeline_run's pull kernel; when the loads are longer (the host link
 * sets the time) the pull kernel, which needs no scatter, is as fast or faster.
 */
pcr_status pcr_pipeline_run_staged(const pcr_layer_io *layers, int32_t n_layers, const pcr_batch *batch,
                                   void *workspace, int64_t workspace_bytes, void *copy_stream,
                                   void *scatter_stream, void *compute_stream, float *timing_ms);

/*
 * pcr_pipeline_run_offload -- the three-stream form (Sec. 5: upload, compute and
 * download streams; Sec. 4.3: offloading a layer starts when its computation
 * ends). As pcr_pipeline_run, and in addition, after layer l's compute,
 * offload_stream waits for it and copies pool blocks off_src[i] of layer l into
 * host blocks off_dst[i] of offload_dst[l] (i < n_off, host arrays, the same list
 * for every layer) with offload_method. offload_dst: host array of n_layers pinned
 * stores. workspace / workspace_bytes: the staging memory of the offload stream
 * when offload_method is PCR_LOAD_DMA_STAGED (else unused, may be NULL / 0).
 * Before its first load the copy stream also waits for the work already queued on
 * offload_stream, so a load never overwrites a pool an earlier offload is still
 * reading. The three streams must differ.
 * timing_ms: NULL, or host float[6*n_layers + 3]; when given the call waits for
 * the last offload and fills, per layer l: [6l] load ms, [6l+1] compute ms,
 * [6l+2] compute-stream wait before the layer, [6l+3] end of the layer's compute
 * and [6l+5] end of its offload (both relative to the pipeline start), [6l+4]
 * offload ms; then [6n] the whole pipeline ms (to the last offload end), [6n+1]
 * the sum of compute ms, [6n+2] the end of the last compute.
 */
pcr_status pcr_pipeline_run_offload(const pcr_layer_io *layers, const pcr_host_kv *offload_dst,
                                    int32_t n_layers, const pcr_batch *batch, const int32_t *off_src,
                                    const int32_t *off_dst, int32_t n_off, pcr_load_method method,
                                    pcr_load_method offload_method, void *workspace, int64_t workspace_bytes,
                                    void *copy_stream, void *compute_stream, void *offload_stream,
                                    float *timing_ms);

/*
 * pcr_pipeline_run_offload_staged -- pcr_pipeline_run_offload with the loads
 * staged as in pcr_pipeline_run_staged: four streams (copy-engine transfers into
 * load_workspace slots on copy_stream, the scatter into the pool on
 * scatter_stream, append and attention on compute_stream, the offload of layer l
 * after its compute on offload_stream with offload_method and offload_workspace).
 * load_workspace follows pcr_pipeline_run_staged's workspace rules;
 * offload_workspace pcr_pipeline_run_offload's; the two must not overlap. Besides
 * the waits of both forms, the first scatter also waits for the work already
 * queued on offload_stream (an earlier offload may still read a pool). The four
 * streams must differ. timing_ms and errors as pcr_pipeline_run_offload; [6l]
 * (load ms) spans the layer's transfers and scatter.
 */
pcr_status pcr_pipeline_run_offload_staged(const pcr_layer_io *layers, const pcr_host_kv *offload_dst,
                                           int32_t n_layers, const pcr_batch *batch, const int32_t *off_src,
                                           const int32_t *off_dst, int32_t n_off, pcr_load_method offload_method,
                                           void *offload_workspace, int64_t offload_workspace_bytes,
                                           void *load_workspace, int64_t load_workspace_bytes, void *copy_stream,
                                           void *scatter_stream, void *compute_stream, void *offload_stream,
                                           float *timing_ms);

/*
 * The SSD tier of the chunk cache (Sec. 4.4 queue-based prefetch and asynchronous
 * write-back; Sec. 5 dedicated prefetch thread). A store is one file of fixed-size
 * chunk slots (chunk id c at byte c * chunk_bytes) served by io_threads host
 * threads in submission order. The file is created (truncated) at open. Buffers
 * belong to the caller and must stay untouched until the chunk's task completes;
 * page-aligned buffers (e.g. pinned host memory) with a page-multiple chunk size
 * bypass the page cache (O_DIRECT). No GPU work is involved.
 *   pcr_store_write_async   queue chunk_bytes from src as chunk chunk_id
 *   pcr_store_read_async    queue a read of chunk chunk_id into dst; PCR_ERR_INVALID_ARG
 *                           if the chunk was never written
 * Tasks of one chunk run one at a time, in submission order: both submit calls
 * first block until the chunk's earlier tasks are done (tasks of other chunks run
 * concurrently on the I/O threads).
 *   pcr_store_wait          block until chunk_id's tasks (or, for chunk_id < 0, all
 *                           tasks) are done; reports the first I/O error, if any
 *   pcr_store_poll          *done = 1 if nothing is pending for chunk_id (or at all)
 *   pcr_store_stats         bytes moved so far; whether the file is open for O_DIRECT;
 *                           and how many page-aligned transfers O_DIRECT refused (host
 *                           memory the GPU driver mapped, such as hipHostMalloc pinned
 *                           memory) and the page cache served instead
 * Any output pointer of pcr_store_stats may be NULL.
 *   pcr_store_close         drain the queue, stop the threads, close the file
 */
typedef struct pcr_chunk_store pcr_chunk_store;
pcr_status pcr_store_open(const char *path, int64_t chunk_bytes, int32_t io_threads, pcr_chunk_store **out);
pcr_status pcr_store_write_async(pcr_chunk_store *store, int64_t chunk_id, const void *src);
pcr_status pcr_store_read_async(pcr_chunk_store *store, int64_t chunk_id, void *dst);
pcr_status pcr_store_wait(pcr_chunk_store *store, int64_t chunk_id);
pcr_status pcr_store_poll(pcr_chunk_store *store, int64_t chunk_id, int32_t *done);
pcr_status pcr_store_stats(pcr_chunk_store *store, int64_t *bytes_read, int64_t *bytes_written, int32_t *direct,
                           int64_t *direct_fallbacks);
pcr_status pcr_store_close(pcr_chunk_store *store);

/* Message of the last failed call on this thread ("" if none). */
const char *pcr_last_error(void);

/* Library version string. */
const char *pcr_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PCR_H_ */
