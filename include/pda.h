/*
 * pda.h -- C interface of the MI355X (gfx950) paged-KV decode-attention library.
 *
 * What it computes. Rollout decoding -- one new token per live sequence per
 * step over a long-tailed mix of sequence lengths -- is the phase of RLVR
 * training whose throughput collapses in the tail (paper Sec. 2.2; decode
 * throughput per GPU in Sec. 6.2, Fig. e2e-conv(c)). Each decode step of the
 * Transformer models it serves (Sec. 1) attends the new token's query to the
 * keys and values cached for its sequence, read through a block table as in
 * the paged KV-cache memory management the paper cites in Sec. 8 (vLLM):
 *
 *     out[b, h, :] = softmax(softmax_scale * K_b q[b, h]) V_b
 *
 * where K_b and V_b hold tokens 0 .. seq_lens[b]-1 of KV head h / G,
 * G = num_q_heads / num_kv_heads (query heads g*G .. g*G+G-1 share KV head g).
 *
 * All entry points are plain C; every pointer argument of
 * pda_paged_decode_attention is a device pointer (HBM) owned by the caller.
 */
#ifndef PDA_H
#define PDA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PDA_VERSION 1

/* Element types. PDA_DTYPE_FP8_E4M3 is the OCP 8-bit E4M3 format without
 * infinities ("e4m3fn": bias 7, max 448, NaN = S.1111.111). */
typedef enum pda_dtype {
  PDA_DTYPE_F32 = 0,
  PDA_DTYPE_BF16 = 1,
  PDA_DTYPE_FP8_E4M3 = 2
} pda_dtype;

/* Return codes. Negative values are errors; pda_last_error() has the text. */
typedef enum pda_status {
  PDA_OK = 0,
  PDA_EINVAL = -1,        /* null pointer, bad size, bad dtype combination      */
  PDA_EUNSUPPORTED = -2,  /* valid but not implemented (head_dim, block size...) */
  PDA_EHIP = -3,          /* a HIP runtime call or a kernel launch failed        */
  PDA_ENOMEM = -4         /* the library's workspace could not be allocated      */
} pda_status;

/* Kernel family. AUTO picks MFMA for bf16/fp8 caches with a GQA group of at
 * least 4 query heads and the vector kernel otherwise. */
typedef enum pda_variant {
  PDA_VARIANT_AUTO = 0,
  PDA_VARIANT_VECTOR = 1, /* VALU dot products with wavefront (DPP) reductions */
  PDA_VARIANT_MFMA = 2    /* bf16 matrix-core QK^T and PV per GQA group        */
} pda_variant;

/* Sizes and element types of one decode step.
 *
 *   q            [num_seqs, num_q_heads, head_dim]            q_dtype, contiguous
 *   k_cache      [num_blocks, num_kv_heads, block_size, head_dim] kv_dtype, contiguous
 *                (token-major tile per (block, KV head))
 *   v_cache      [num_blocks, num_kv_heads, head_dim, block_size] kv_dtype, contiguous
 *                (dim-major tile per (block, KV head))
 *   block_table  [num_seqs, max_blocks_per_seq] int32 physical block ids; entry j
 *                of row b holds tokens 16j .. 16j+15 of sequence b; entries at or
 *                past ceil(seq_lens[b] / 16) are never read
 *   seq_lens     [num_seqs] int32, 0 <= seq_lens[b] <= max_seq_len
 *   kv_scales    [2, num_blocks, num_kv_heads] fp32 dequantisation scales, index 0
 *                for K and 1 for V; required for fp8 caches, ignored otherwise
 *   out          [num_seqs, num_q_heads, head_dim] out_dtype, contiguous
 *
 * q, k_cache, v_cache and out must be 16-byte aligned (the kernels move them
 * in 16-byte units); block_table, seq_lens and kv_scales 4-byte aligned.
 * Misaligned pointers are rejected with PDA_EINVAL.
 *
 * max_seq_len is a host-side upper bound on every seq_lens[b] (0 means
 * max_blocks_per_seq * block_size). Lengths above it, above
 * max_blocks_per_seq * block_size, or below 0 are clamped into range on the
 * device and reported by pda_read_device_status(); so are block-table entries
 * outside [0, num_blocks), whose blocks are then skipped.
 */
typedef struct pda_problem {
  int32_t num_seqs;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;            /* 64 or 128 */
  int32_t block_size;          /* tokens per KV block: 16 */
  int32_t max_blocks_per_seq;  /* row length (and stride) of block_table */
  int64_t num_blocks;          /* physical blocks in k_cache / v_cache */
  int32_t max_seq_len;
  int32_t q_dtype;             /* pda_dtype: F32 or BF16 */
  int32_t kv_dtype;            /* pda_dtype: F32 (needs F32 q), BF16 or FP8_E4M3 (need BF16 q) */
  int32_t out_dtype;           /* pda_dtype of out: q_dtype or F32 (accumulation stays fp32) */
  int32_t q_tokens;            /* query tokens per sequence; 0 or 1: one (a decode step). Q > 1
                                  (speculative verification of drafted tokens, named among the RLVR
                                  rollout strategies of the paper's Sec. 1): q and out are
                                  [B, Q, Hq, D], the cache already holds the Q new tokens as the
                                  sequence's last Q, and query token i attends causally to tokens
                                  0 .. L - Q + i (zeros if none). Needs the MFMA kernel (bf16 or fp8
                                  cache) and Q * G <= 32. */
} pda_problem;

/* Optional tuning knobs; pass NULL for the defaults (all zero). */
typedef struct pda_options {
  int32_t variant;              /* pda_variant */
  int32_t waves_per_cu;         /* persistent waves launched per compute unit; 0 = auto */
  int32_t min_blocks_per_wave;  /* no chunk of work is smaller than this many block-heads
                                   (16 tokens of one KV head); 0 = auto (8) */
  int32_t chunks_per_wave;      /* 1 = static split (one equal chunk per wave); k > 1 = up to
                                   k chunks per wave, handed out dynamically; 0 = default (1) */
  int32_t min_blocks_per_chunk; /* a dynamic split makes no chunk smaller than this many
                                   block-heads; 0 = auto (512 KiB of K and V) */
} pda_options;

/* Host-side plan of one call: what pda_paged_decode_attention would launch. */
typedef struct pda_plan_info {
  int32_t variant;             /* the kernel family that runs (never AUTO) */
  int32_t waves;               /* persistent waves (workgroups of up to 4 independent waves) */
  int32_t group_size;          /* G = num_q_heads / num_kv_heads */
  int32_t chunks_max;          /* most chunks the split can cut (waves * chunks_per_wave) */
  int64_t workspace_bytes;     /* library-owned device workspace this call needs */
} pda_plan_info;

/*
 * One batched decode-attention step, enqueued on `stream` (a hipStream_t; NULL
 * is the null stream). Asynchronous: results are valid once the stream has
 * reached this point. The step's KV blocks (16 tokens of one KV head each,
 * plus a small start cost per sequence and KV head counted in the same units)
 * are cut into equal chunks that persistent waves take in turn (each wave its
 * own first chunk, the rest in arrival order); a sequence split between
 * chunks is finished by a log-sum-exp combine kernel on the same stream. The result does not depend
 * on which wave ran which chunk: repeated calls give identical output.
 *
 * Ownership: the caller owns every buffer; the library keeps no pointer to
 * them after returning. It owns one device workspace per (device, stream),
 * grown on demand (growth synchronises that stream) and released by
 * pda_release_workspaces().
 *
 * HIP graphs: once the stream's workspace is large enough (a call of the same
 * or a larger size has run on it), a call enqueues kernel launches only, so it
 * can be captured into a graph and replayed; the captured launches keep the
 * pointers and sizes of the capture, and inputs may change in place between
 * replays. A call that would grow the workspace during capture returns
 * PDA_EINVAL instead of allocating; growth after a capture keeps the old
 * allocation for the graph until pda_release_workspaces(), after which no
 * graph captured before may be replayed. This holds for every call below.
 *
 * Errors: all argument checks run on the host before any HIP call, so invalid
 * arguments return PDA_EINVAL / PDA_EUNSUPPORTED without touching a device.
 * Returns PDA_OK once the kernels are enqueued.
 *
 * Thread safety: calls on different streams may run concurrently; calls on
 * one stream from several threads are serialised by an internal lock.
 */
int pda_paged_decode_attention(const void* q,
                               const void* k_cache,
                               const void* v_cache,
                               const int32_t* block_table,
                               const int32_t* seq_lens,
                               const float* kv_scales,
                               void* out,
                               float softmax_scale,
                               const pda_problem* problem,
                               const pda_options* options,
                               hipStream_t stream);

/*
 * For callers that cannot allocate device memory: code being captured into a
 * HIP graph before any eager call has sized a workspace, tight serving loops,
 * harnesses that forbid hipMalloc. The same decode step as
 * pda_paged_decode_attention, with the same arguments, kernels and result
 * (bitwise), but its workspace (partial results, per-sequence prefix sums,
 * chunk counter, status word) is a fixed device array of PDA_NOALLOC_SCRATCH_BYTES
 * (32 MiB) compiled into the library: each device the library runs on holds
 * its own copy from load until the process ends. The call allocates nothing:
 * no hipMalloc, hipFree or allocating library routine, on any call.
 *
 * Limit: a call whose workspace (pda_plan_info.workspace_bytes) exceeds the
 * array returns PDA_EINVAL with the size it needed; at the default split that
 * is about 25 MiB for 512 sequences x 8 KV heads x 8 query heads per KV head
 * (more waves per CU, dynamic chunks or wider query groups need more).
 *
 * Sharing: every call on a device uses that device's one array, and the
 * array keeps the last call's contents. Calls that overlap on one device
 * (different streams, or threads without ordering between them) race on it
 * and may give wrong results; order them on one stream. Calls on one stream
 * from several threads are serialised by an internal lock, as are calls on
 * different devices. The chunk counter starts at zero (the array is
 * zero-initialised at load) and the combine kernel re-zeroes it after every
 * call. Status bits go to the array's status word, which
 * pda_read_device_status(stream) reads and clears too (after waiting for
 * `stream` only).
 *
 * Errors as for pda_paged_decode_attention, plus PDA_EINVAL for the size limit
 * above. Capturable into a HIP graph from the first call.
 */
#define PDA_NOALLOC_SCRATCH_BYTES (32LL << 20)
int pda_paged_decode_attention_noalloc(const void* q,
                                       const void* k_cache,
                                       const void* v_cache,
                                       const int32_t* block_table,
                                       const int32_t* seq_lens,
                                       const float* kv_scales,
                                       void* out,
                                       float softmax_scale,
                                       const pda_problem* problem,
                                       const pda_options* options,
                                       hipStream_t stream);

/* Validate `problem` / `options` and describe the launch, on the host only
 * (no HIP call). `num_compute_units` sizes the persistent grid (MI355X: 256).
 * With options.waves_per_cu = 0 the launch takes the decode kernel's
 * occupancy (at most 8 waves per CU), which only the device knows: `waves`,
 * `chunks_max` and `workspace_bytes` are then upper bounds (8 waves per CU).
 * Returns the same error codes as pda_paged_decode_attention. */
int pda_query_plan(const pda_problem* problem,
                   const pda_options* options,
                   float softmax_scale,
                   int32_t num_compute_units,
                   pda_plan_info* info);

/*
 * The same decode step for batches of equal-size groups whose members share
 * leading KV blocks: GRPO-style rollouts, where every prompt is sampled
 * group_size times and the samples' block tables start with the prompt's
 * blocks. Sequences g*group_size .. g*group_size + group_size - 1 form group g,
 * and shared_blocks[g] (device, [num_seqs / group_size] int32) bounds how many
 * leading 16-token blocks its members share. The result is the same attention
 * pda_paged_decode_attention computes; only the work differs: each shared
 * block is read once for up to 16 query heads of several members (ceil(
 * group_size * G / 16) reads instead of group_size). GRPO, one of the RLVR
 * objectives of the paper's Sec. 2.3 and the setup of its Sec. 6.3
 * simulation, samples a group of responses for every prompt, so a rollout
 * batch is made of such groups.
 *
 * The library verifies the bound on the device: a group shares at most
 * shared_blocks[g] blocks, at most every member's full blocks, and only as
 * long as every member's block-table row holds the same block ids; a bound that
 * ids contradict sets status bit 4 (see pda_read_device_status). A wrong bound
 * therefore costs speed, never correctness.
 *
 * Errors as for pda_paged_decode_attention, and PDA_EINVAL if group_size < 1,
 * num_seqs is not a multiple of group_size or shared_blocks is NULL;
 * PDA_EUNSUPPORTED for an f32 KV cache or options.variant = VECTOR (the
 * shared-prefix path runs on the MFMA kernel).
 */
int pda_paged_decode_attention_shared_prefix(const void* q,
                                             const void* k_cache,
                                             const void* v_cache,
                                             const int32_t* block_table,
                                             const int32_t* seq_lens,
                                             const float* kv_scales,
                                             void* out,
                                             float softmax_scale,
                                             int32_t group_size,
                                             const int32_t* shared_blocks,
                                             const pda_problem* problem,
                                             const pda_options* options,
                                             hipStream_t stream);

/* pda_query_plan for pda_paged_decode_attention_shared_prefix with this group_size. */
int pda_query_plan_shared_prefix(const pda_problem* problem,
                                 const pda_options* options,
                                 float softmax_scale,
                                 int32_t group_size,
                                 int32_t num_compute_units,
                                 pda_plan_info* info);

/* Shapes and dtypes of one KV append (see pda_paged_kv_append). */
typedef struct pda_append_problem {
  int32_t num_seqs;            /* B */
  int32_t num_kv_heads;        /* Hkv */
  int32_t head_dim;            /* D: 64 or 128 */
  int32_t block_size;          /* tokens per KV block: 16 */
  int32_t max_blocks_per_seq;  /* block_table row stride */
  int64_t num_blocks;          /* NB */
  int32_t new_dtype;           /* k_new / v_new: PDA_DTYPE_F32 or PDA_DTYPE_BF16 */
  int32_t kv_dtype;            /* cache: PDA_DTYPE_F32, PDA_DTYPE_BF16 or PDA_DTYPE_FP8_E4M3 */
} pda_append_problem;

/*
 * The step before attention in every decode step (the paper's Sec. 2.2 rollout
 * decoding, over the paged cache of the vLLM work cited in its Sec. 8): write
 * each sequence's new key and value into its paged cache, enqueued on
 * `stream`.
 *
 *   k_new, v_new  [B, Hkv, D] device, new_dtype (finite values)
 *   k_cache       [NB, Hkv, 16, D], v_cache [NB, Hkv, D, 16]: the layouts
 *                 pda_paged_decode_attention reads
 *   kv_scales     [2, NB, Hkv] fp32 (fp8 caches; NULL otherwise), read and written
 *   block_table   [B, max_blocks_per_seq] int32
 *   positions     [B] int32 device: index of the new token (the sequence's
 *                 length before the append); a negative position skips the
 *                 sequence
 *
 * Token t of sequence b goes to block block_table[b, t / 16], slot t % 16: a
 * row of the K tile and a column of the V tile, rounded to nearest even for a
 * bf16 cache. An fp8 (E4M3) cache keeps each (block, KV head) tile's K and V
 * scales at max(amax / 448, 2^-126) over the tokens written to the tile so
 * far: a token whose amax exceeds 448 * scale raises the scale to its own
 * amax / 448 and re-encodes the tile's earlier codes (decoded value * old /
 * new scale); slot 0 starts a fresh scale. A full tile therefore ends with its
 * amax scale, as in a per-tile quantisation. All code decisions are float32
 * steps (correctly rounded division), encoding rounds to nearest even after
 * clamping to +-448.
 *
 * A position at or past 16 * max_blocks_per_seq, or a block-table entry
 * outside [0, num_blocks), skips that sequence and sets status bit 1 or 2
 * (pda_read_device_status). Two sequences writing the same (block, slot) in
 * one call race. For an fp8 cache the unit of a write is the whole (block, KV
 * head) tile: a new token may raise the tile's K and V scales and re-encode
 * the tile's earlier codes, so two sequences of one call must not append into
 * the same block at all, not even into different slots. Sequences normally
 * append to private blocks (a shared prompt's blocks are full and read-only).
 *
 * Errors: all checks run on the host before any HIP call: PDA_EINVAL for bad
 * sizes, dtypes or NULL pointers, PDA_EUNSUPPORTED for head_dim not in {64,
 * 128} or block_size != 16. Uses the stream's workspace (status word).
 */
int pda_paged_kv_append(const void* k_new,
                        const void* v_new,
                        void* k_cache,
                        void* v_cache,
                        float* kv_scales,
                        const int32_t* block_table,
                        const int32_t* positions,
                        const pda_append_problem* problem,
                        hipStream_t stream);

/* Shapes and dtypes of one variable-length prefill (see pda_paged_prefill_attention). */
typedef struct pda_prefill_problem {
  int32_t num_seqs;            /* B */
  int32_t num_tokens;          /* T: packed query rows of q and out */
  int32_t num_q_heads;         /* Hq */
  int32_t num_kv_heads;        /* Hkv; G = Hq / Hkv <= 16 */
  int32_t head_dim;            /* D: 64 or 128 */
  int32_t block_size;          /* tokens per KV block: 16 */
  int32_t max_blocks_per_seq;  /* block_table row stride */
  int64_t num_blocks;          /* NB */
  int32_t max_seq_len;         /* host bound on seq_lens (0 = max_blocks_per_seq * 16) */
  int32_t q_dtype;             /* PDA_DTYPE_BF16 */
  int32_t kv_dtype;            /* PDA_DTYPE_BF16 or PDA_DTYPE_FP8_E4M3 */
  int32_t out_dtype;           /* PDA_DTYPE_BF16 or PDA_DTYPE_F32 */
} pda_prefill_problem;

/*
 * Causal attention of many query tokens per sequence over the paged cache,
 * enqueued on `stream`: the log-prob forward of RLVR training (the
 * compute_log_prob phase timed in the paper's Table 2, Sec. 6.3; a forward call
 * of the remote execution interface of its Sec. 4.2) and chunked prefill. The
 * cache already holds every token's key and value (pda_paged_kv_append, or the
 * caller's own writes).
 *
 *   q            [T, Hq, D] bf16: rows q_offsets[b] .. q_offsets[b+1]-1 are the
 *                last n_b = q_offsets[b+1] - q_offsets[b] tokens of sequence b
 *   q_offsets    [B + 1] int32 device, non-decreasing, q_offsets[0] >= 0,
 *                q_offsets[B] <= T
 *   k_cache, v_cache, block_table, seq_lens, kv_scales: as for
 *                pda_paged_decode_attention (seq_lens[b] = L_b, all cached tokens)
 *   out          [T, Hq, D] out_dtype; rows outside every sequence are not written
 *
 * Query token i of sequence b sits at position L_b - n_b + i and attends to
 * tokens 0 .. L_b - n_b + i of its sequence (softmax_scale on the logits, KV
 * head h / G); a token at a negative position (n_b > L_b) gets zeros. Every
 * output row is computed by one workgroup with no split of the keys, so the
 * result does not depend on the launch order.
 *
 * Precision: q . k in bf16 products with fp32 sums; the softmax weights (at
 * most 2^8 after the running-max shift) and V (fp8: code times V scale) enter
 * the P . V product as fp16 (11 significant bits; bf16 V converts exactly),
 * accumulated in fp32. A live V value beyond +-65504 saturates (status bit 16).
 *
 * Image: each call first converts every cache tile that its sequences read
 * into the stream's workspace, in the products' operand types (V to fp16, and
 * for an fp8 cache K codes to bf16), indexed like the cache; the attention
 * kernel then copies tiles from that image straight into LDS. The image takes
 * num_blocks * num_kv_heads * 16 * head_dim * 2 bytes (twice that for an fp8
 * cache). When that exceeds the environment variable PDA_PREFILL_IMAGE_MAX_MB
 * (MiB, read on every call; default 8192), when a stream being captured into a
 * HIP graph has too small a workspace for it, or when its allocation fails, the
 * kernel converts each tile in registers instead. Both ways give bit-identical
 * outputs.
 *
 * Device-checked: lengths are clamped as in decode (status bit 1), block-table
 * entries outside [0, num_blocks) are skipped (bit 2), and offsets that are not
 * non-decreasing within [0, T] make the call write nothing (bit 8).
 *
 * Errors: all checks run on the host before any HIP call: PDA_EINVAL for bad
 * sizes, dtypes, NULL pointers or misaligned ones (q, the caches and out need
 * 16 bytes, the int32 and f32 arrays 4), or more than INT32_MAX / 8 work units
 * (tiles of 256 / G query tokens times KV heads); PDA_EUNSUPPORTED for
 * head_dim not in {64, 128}, block_size != 16, G > 16, or an f32 cache. Uses
 * the stream's workspace: 16 bytes per work item of 256 / G query tokens, plus
 * the image described above.
 */
int pda_paged_prefill_attention(const void* q,
                                const int32_t* q_offsets,
                                const void* k_cache,
                                const void* v_cache,
                                const int32_t* block_table,
                                const int32_t* seq_lens,
                                const float* kv_scales,
                                void* out,
                                float softmax_scale,
                                const pda_prefill_problem* problem,
                                hipStream_t stream);

/* Wait for `stream`, then return (and clear) the device-side status bits that
 * calls on it recorded (and those in the fixed scratch of
 * pda_paged_decode_attention_noalloc, once it has run on the device): 1 = a
 * sequence length was clamped, 2 = a block-table
 * entry outside [0, num_blocks) was skipped, 4 = a group's members share fewer
 * leading blocks than shared_blocks declared, 8 = prefill q_offsets were not
 * non-decreasing within [0, T], 16 = a prefill V value outside the fp16 range
 * saturated. 0 when clean; negative on error. */
int pda_read_device_status(hipStream_t stream);

/* Free every workspace the library holds (waits for the owning streams). */
int pda_release_workspaces(void);

/* Text of the last error on the calling thread ("" if none). */
const char* pda_last_error(void);

/* PDA_VERSION of the built library. */
int pda_version(void);

#ifdef __cplusplus
}  /* extern "C" */
#endif

#endif  /* PDA_H */
