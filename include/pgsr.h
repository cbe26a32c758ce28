/*
 * pgsr.h -- C ABI of the selective-replay hot path on MI355X (gfx950).
 *
 * The paper ("Forgetting Without Restarting: Execution-State Unlearning for
 * Stateful LLM Agents") states forgetting as splicing a deterministic
 * transition system R_t = F(R_{t-1}, o_t) (Section 3.1, Eq. (1)): the state up to
 * the injection step tau is shared with the counterfactual run (Lemma 1), so a
 * checkpoint restore is a crop of the KV cache to tau - 1 (Section 3.4 (b);
 * Algorithm 1, restore step) and the T - tau + 1 sanitized transitions after it
 * are replayed (Algorithm 1, replay loop; Theorem 1), which is optimal
 * (Corollary 1).  A full reset replays all T transitions (baseline B5,
 * Section 4.1).  Replayed content that is fixed in the counterfactual world is
 * re-materialised by prefill (Section 3.2, after Lemma 2), which is what
 * pgsr_replay_prefill computes.
 *
 * Memory model.  Every device pointer is owned by the caller (allocated, e.g.,
 * as torch tensors), must stay valid for the pool's lifetime and is never
 * freed or reallocated here.  The library allocates no device memory (the
 * checked build below: one 4-byte flag per pool, at pool creation).  It keeps
 * a HOST mirror of per-sequence length and block count and of the free-list
 * top, updated at call time in enqueue order; one pool must not be used from
 * two host threads at once.
 *
 * Device layout (elements of the pool dtype -- 4, 2 or 1 bytes -- row-major):
 *   k_cache      [n_layers][n_blocks][n_kv_heads][block_size][head_dim]
 *   v_cache      [n_layers][n_blocks][n_kv_heads][head_dim][block_size]
 *                (values are stored transposed inside each block: the
 *                 attention kernels read V along the key axis)
 *   block_tables int32 [max_seqs][max_blocks_per_seq], -1 = no block
 *   seq_lens     int32 [max_seqs]          committed tokens per sequence
 *   free_list    int32 [n_blocks]          LIFO stack of free block ids
 *   free_top     int32 [1]                 stack height
 *   ref_counts   int32 [n_blocks]          table entries naming each block
 * Logical token p of sequence s lives in block block_tables[s][p / B] at
 * slot p % B.  Rows may share blocks after pgsr_kv_fork (copy-on-write): a
 * block is free exactly when its count is 0.  A sequence's slots at or beyond its length hold unspecified
 * data (possibly NaN) and are never read.
 *
 * Errors.  Every call returns a status.  Arguments are validated against the
 * host mirror before anything is enqueued: on PGSR_EINVAL / PGSR_ERANGE /
 * PGSR_ENOMEM / PGSR_EUNSUPPORTED nothing was enqueued and neither the mirror
 * nor device state changed.  PGSR_EHIP means a HIP call failed after
 * validation; device state is then undefined and the pool must be re-created.
 * pgsr_last_error() describes the most recent failure on the calling thread.
 *
 * Checked build.  The same sources compiled with PGSR_CHECKED
 * (lib/libpgsr_checked.so, same ABI) validate on the device every block id
 * they read from block_tables or free_list before it addresses the cache, the
 * counts or the stack.  Only device metadata written behind the library's back
 * can hold an id outside [0, n_blocks); the checked build then uses block 0
 * instead, finishes the call's launches, waits for them, and returns
 * PGSR_ERANGE from pgsr_kv_crop, pgsr_kv_fork and the prefill calls (device
 * state is then undefined, as after PGSR_EHIP).  Because of that wait, its
 * calls synchronise the stream; it is a debugging aid, not the fast path.
 *
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  Every call
 * only enqueues work and returns without synchronising, except
 * pgsr_pool_create and pgsr_pool_refresh, which block.
 */
#ifndef PGSR_H
#define PGSR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    PGSR_OK = 0,
    PGSR_EINVAL = 1,        /* bad argument: null pointer, bad id, duplicate sequence */
    PGSR_ERANGE = 2,        /* a length outside what the sequence or its table row allows */
    PGSR_ENOMEM = 3,        /* the free list holds too few blocks */
    PGSR_EUNSUPPORTED = 4,  /* a geometry or dtype with no kernel */
    PGSR_EHIP = 5,          /* a HIP runtime call or launch failed */
    PGSR_ENOENT = 6         /* front-end: the target never entered, or no checkpoint precedes tau */
};

/* Pool dtypes.  PGSR_FP8_E4M3 stores K/V as 1-byte OCP E4M3 codes with
 * per-layer scales (pgsr_pool_set_kv_scales); its q, k, v inputs and o
 * outputs are bf16 and attention runs in bf16 on the widened codes. */
enum { PGSR_F32 = 0, PGSR_BF16 = 1, PGSR_FP8_E4M3 = 2 };

/* flags */
#define PGSR_COMMIT 1u        /* replay: advance each sequence's length by its q_len */
#define PGSR_POISON 2u        /* crop: fill released slots with NaN (debug aid) */

typedef struct pgsr_pool pgsr_pool;

/* Text of the last failure on this thread; "" if none.  Valid until the next
 * call on this thread. */
const char *pgsr_last_error(void);

/* Library ABI version (increments on incompatible changes). */
int pgsr_abi_version(void);

/*
 * Create a pool over caller-owned device memory and initialise its device
 * state: every table entry -1, every length 0, every count 0, free_list = the
 * initial stack, free_top = n_blocks.  init_free_order (HOST, nullable, n_blocks entries) is
 * the stack from bottom to top and must be a permutation of 0 .. n_blocks-1;
 * NULL means n_blocks-1 .. 0, so pops yield 0, 1, 2, ....  The KV caches are
 * not touched.  workspace (device, nullable) is scratch for split-key partial
 * results, workspace_bytes long (see pgsr_workspace_bytes); NULL disables
 * key splitting.  Supported: dtype PGSR_F32, PGSR_BF16 or PGSR_FP8_E4M3,
 * head_dim 64 or 128, block_size 16, 32 or 64, n_q_heads a multiple of
 * n_kv_heads (bf16 and fp8: at most 32 query heads per KV head, any such
 * group, e.g. 7 for 28 / 4 heads).  An FP8 pool starts with every scale 1.
 * Blocks.
 */
int pgsr_pool_create(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                     int32_t block_size, int32_t dtype, int32_t n_blocks, int32_t max_seqs,
                     int32_t max_blocks_per_seq, void *k_cache, void *v_cache,
                     int32_t *block_tables, int32_t *seq_lens, int32_t *free_list,
                     int32_t *free_top, int32_t *ref_counts, void *workspace,
                     size_t workspace_bytes, const int32_t *init_free_order, void *stream,
                     pgsr_pool **out);

/*
 * FP8 KV cache (a storage variant of the cache that Algorithm 1 crops and
 * appends to; the paper keeps the cache at model precision): k_scales and
 * v_scales (HOST, n_layers positive normal floats each) become the layers'
 * scales for later appends and reads.  An appended bf16 value x of layer l is
 * stored as the E4M3 code of the correctly rounded fp32 quotient x / scale,
 * rounded to nearest even, magnitudes past 448 saturating to 448, NaN kept
 * NaN; attention reads code * scale.  Codes already in the cache keep the
 * scale they were written with only if the scale does not change: set the
 * scales before the first append.  PGSR_EINVAL for a non-FP8 pool or a bad
 * scale (then nothing changes).  Host only, no device work.
 */
int pgsr_pool_set_kv_scales(pgsr_pool *pool, const float *k_scales, const float *v_scales);

/* Release the host object; device memory is the caller's. NULL is a no-op. */
int pgsr_pool_destroy(pgsr_pool *pool);

/* Re-read the host mirror from device state (blocking).  For callers that
 * restore block_tables / seq_lens / free_list / free_top / ref_counts
 * themselves, e.g. by copying a saved pre-crop state back; a row's block count
 * is taken as the number of leading non-negative entries. */
int pgsr_pool_refresh(pgsr_pool *pool, void *stream);

/* Host-mirror queries (no device access). */
int pgsr_seq_len(const pgsr_pool *pool, int32_t seq, int32_t *len_out);
int pgsr_free_blocks(const pgsr_pool *pool, int32_t *n_out);

/* Bytes of workspace that let a replay of up to max_total_q query tokens use
 * up to max_splits key splits. */
size_t pgsr_workspace_bytes(int32_t n_q_heads, int32_t head_dim, int64_t max_total_q,
                            int32_t max_splits);

/*
 * Restore = crop (Algorithm 1, restore step; Section 3.4 (b); Lemma 1): for
 * each i, keep the first new_lens[i] tokens of sequence seqs[i]
 * (0 <= new_lens[i] <= its length).  Table entries from ceil(new_len / B) on
 * become -1 and each such block's count drops by 1; blocks whose count reaches
 * 0 are pushed onto the free list, sequences in call order, ascending logical
 * block within a sequence (without forks every released block is pushed); a
 * crop to the current length is a no-op and a crop to 0 releases every entry.  KV data of the kept
 * tokens is not touched.  seqs and new_lens are HOST arrays of n entries; a
 * duplicate sequence is PGSR_EINVAL.  flags: 0 or PGSR_POISON.
 * All-or-nothing.
 */
int pgsr_kv_crop(pgsr_pool *pool, int32_t n, const int32_t *seqs, const int32_t *new_lens,
                 unsigned flags, void *stream);

/*
 * Copy-on-write fork (every method branches from the same contaminated base,
 * Section 4.1): for each i, the EMPTY sequence dsts[i] (length 0, no blocks)
 * takes the table row and length of srcs[i]; no KV data moves, and each shared
 * block's count grows by 1.  Later crops of either row release only their own
 * references, and the first write into a shared partial tail block copies it
 * (see pgsr_replay_prefill).  srcs, dsts: HOST arrays of n; a target that is
 * not empty, appears twice or is also a source is PGSR_EINVAL.  All-or-nothing.
 */
int pgsr_kv_fork(pgsr_pool *pool, int32_t n, const int32_t *srcs, const int32_t *dsts,
                 void *stream);

/*
 * One layer of F over the sanitized suffix, prefill form (Algorithm 1, replay
 * loop; Theorem 1; re-materialisation by prefill, Section 3.2 after Lemma 2).
 * For each i, with P_i the committed length of seqs[i] and S_i = q_lens[i]:
 *   1. blocks for positions P_i .. P_i+S_i-1 are popped from the free list when
 *      the row holds fewer (so the first layer of a step reserves them); if
 *      the partial tail block (P_i mod B != 0) is shared with another row, a
 *      private block is popped first and receives its slots 0 .. P_i mod B - 1
 *      of every layer (copy-on-write; the shared block's count drops by 1);
 *   2. the S_i new keys/values are written to positions P_i .. P_i+S_i-1 of
 *      `layer` (filling the partial tail block first);
 *   3. o receives, for the query at absolute position p = P_i + t and query
 *      head h (KV head h / (n_q_heads / n_kv_heads)), softmax attention over
 *      keys 0 .. p:  o = sum_j softmax_j(softmax_scale * q.k_j) v_j.
 * q, o : [sum S_i][n_q_heads][head_dim];  k, v : [sum S_i][n_kv_heads][head_dim],
 * device, pool dtype (bf16 for an FP8 pool, whose k_j and v_j are the
 * stored codes times the layer's scales), packed in seqs order.  seqs,
 * q_lens: HOST arrays.
 * flags & PGSR_COMMIT adds S_i to each length (set it on the last layer of a
 * step) and sum S_i to *recomputed_tokens (HOST, nullable) -- the count of
 * Corollary 1.  Outputs are bitwise reproducible run to run.  On a pool
 * without a workspace they depend only on each query's absolute position, not
 * on how the suffix is batched.  With a workspace, a call that would leave
 * compute units idle splits keys over several workgroups, and a call whose
 * sequences all have at most 32 / (n_q_heads / n_kv_heads) query tokens (a
 * decode step) runs a decode kernel; both round in another order, so their
 * bits depend on the call's shape as well.
 */
int pgsr_replay_prefill(pgsr_pool *pool, int32_t layer, int32_t n, const int32_t *seqs,
                        const int32_t *q_lens, const void *q, const void *k, const void *v,
                        void *o, float softmax_scale, unsigned flags,
                        int64_t *recomputed_tokens, void *stream);

/*
 * Algorithm 1's restore step followed by the first layer of its replay loop,
 * in one call (Section 3.4 (b): restoring a checkpoint is a crop; Theorem 1:
 * replay from there).  The same device state, outputs and recompute count,
 * bit for bit, as pgsr_kv_crop(pool, n, seqs, restore_lens, 0, stream)
 * followed by pgsr_replay_prefill(pool, layer, n, seqs, q_lens, ...), but
 * validated together on the host mirror (all-or-nothing across both: the
 * replay is checked against the state the crop leaves) and, where it applies
 * (bf16 pool, at most 16 sequences each with query tokens, at most 512
 * appended blocks, no kept partial tail block shared with another row), with
 * the crop's device work in the append launch: one launch and one host call
 * fewer between the restore and the replay.  seqs, restore_lens, q_lens: HOST
 * arrays of n; the other arguments as for pgsr_replay_prefill.
 */
int pgsr_restore_replay_prefill(pgsr_pool *pool, int32_t layer, int32_t n, const int32_t *seqs,
                                const int32_t *restore_lens, const int32_t *q_lens, const void *q,
                                const void *k, const void *v, void *o, float softmax_scale,
                                unsigned flags, int64_t *recomputed_tokens, void *stream);

/*
 * pgsr_replay_prefill for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  Same arguments, kernels and results as pgsr_replay_prefill on
 * a pool whose workspace were scratch_bytes large (bitwise), except that the
 * split-key and decode partials live in a device array the library holds for
 * the whole process on each GPU it runs on, PGSR_STATIC_SCRATCH_BYTES (64 MiB)
 * large; the pool's own workspace is not used.  scratch_bytes bounds the
 * partials of this call (pgsr_workspace_bytes sizes it: up to max_splits
 * splits of up to max_total_q query tokens); 0 runs without splits;
 * scratch_bytes > PGSR_STATIC_SCRATCH_BYTES is PGSR_ERANGE and changes
 * nothing.  No hipMalloc, hipFree or other allocation of device memory.
 * Every call on one GPU shares that GPU's array and leaves its contents
 * there: calls whose work overlaps on one GPU (two streams, two host threads)
 * race.  The partials need no clearing: each call writes every entry it reads.
 */
#define PGSR_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int pgsr_replay_prefill_static(pgsr_pool *pool, int32_t layer, int32_t n, const int32_t *seqs,
                               const int32_t *q_lens, const void *q, const void *k, const void *v,
                               void *o, float softmax_scale, unsigned flags, size_t scratch_bytes,
                               int64_t *recomputed_tokens, void *stream);

/*
 * Full reset (baseline B5, Section 4.1; T invocations of F, Corollary 1): on
 * layer 0 the sequences are first cropped to 0, then the whole sanitized
 * trajectory (lens[i] tokens) is replayed exactly as pgsr_replay_prefill does
 * with P_i = 0.  Same arguments and validation; all-or-nothing.
 */
int pgsr_full_reset_prefill(pgsr_pool *pool, int32_t layer, int32_t n, const int32_t *seqs,
                            const int32_t *lens, const void *q, const void *k, const void *v,
                            void *o, float softmax_scale, unsigned flags,
                            int64_t *recomputed_tokens, void *stream);

/*
 * Kernel timing for profiling tools.  With timing on, every replay / full-reset
 * call records HIP events on its stream around its append launches and around
 * its attention launches (a few microseconds of overhead per call).
 * pgsr_pool_last_times waits for the most recent such call's events and
 * returns the GPU time of its append and attention kernels in milliseconds.
 */
int pgsr_pool_enable_timing(pgsr_pool *pool, int on);
int pgsr_pool_last_times(pgsr_pool *pool, float *append_ms, float *attention_ms);

/*
 * Shader-clock probe for profiling tools.  `buf` is caller-owned device memory
 * of `bytes` bytes (NULL or 0 turns the probe off); it must outlive its use.
 * While timing is on (pgsr_pool_enable_timing) and a buffer is set, a
 * replay / full-reset call that runs the pipelined bf16 prefill kernel zeroes
 * the buffer and then, for each of its first bytes / 32 workgroups, writes four
 * uint64: the shader-cycle counter (s_memtime) and the constant-rate reference
 * counter (s_memrealtime) at the workgroup's start and at its end.  A call
 * with several attention launches keeps only its last one.
 * pgsr_pool_last_clock waits for the stream, reads the buffer back and
 * returns the mean shader clock over those workgroups in GHz (shader cycles
 * over reference ticks times the reference rate), the summed cycles and the
 * summed reference ticks; EINVAL when no timed launch wrote the probe.
 */
int pgsr_pool_set_clock_buffer(pgsr_pool *pool, void *buf, size_t bytes);
int pgsr_pool_last_clock(pgsr_pool *pool, void *stream, double *ghz, int64_t *cycles, int64_t *ticks);

/*
 * Choice of the bf16 prefill attention kernel (Algorithm 1 replay loop,
 * prefill form).  PGSR_PREFILL_AUTO (the default) runs, for a bf16 pool with
 * head_dim 128 and a GQA group dividing 32, the wide kernel (one wave per
 * SIMD, 64 query rows per wave, global->LDS tile loads) when the pool has
 * 16-token blocks, n_blocks * n_kv_heads * 4 KB <= 4 GB and no sequence of
 * the call reaches more than 130816 keys (prefix + suffix), else the
 * software-pipelined kernel (two waves per SIMD, 32 query rows per wave);
 * every other call runs the four-wave kernel.  PGSR_PREFILL_PIPELINED skips
 * the wide kernel; PGSR_PREFILL_FOUR_WAVE runs the four-wave kernel for every
 * call.  All give identical bits for every query row; the option only moves
 * time.  Host only, no device work; EINVAL for another value.
 */
enum { PGSR_PREFILL_AUTO = 0, PGSR_PREFILL_FOUR_WAVE = 1, PGSR_PREFILL_PIPELINED = 2 };
int pgsr_pool_set_prefill_kernel(pgsr_pool *pool, int kind);

/*
 * Dense projection of the stacked-layer transition F (theta in Eq. (1)):
 * Y[m][n] = sum_k X[m][k] * W[n][k] (+ R[m][n] when R != NULL), i.e. Y = X W^T
 * with W in the linear-layer layout [n][k]; bf16 row-major device arrays,
 * fp32 accumulation, one round-to-nearest-even store.  R may alias Y.
 * m, n, k >= 0; n and k must be multiples of 8.  Rows of Y are computed
 * independently with a fixed accumulation order (no split over k).
 */
int pgsr_gemm_bf16(int32_t m, int32_t n, int32_t k, const void *x, const void *w,
                   const void *r, void *y, void *stream);

/*
 * Elementwise steps of a full decoder layer around the projections (F of
 * Eq. (1) at the real geometries; the layer itself follows the public
 * architecture of the model families the paper runs).  bf16 device arrays,
 * row-major, fp32 arithmetic, one round-to-nearest-even per stored value.
 *
 * RMSNorm: y[r] = x[r] / sqrt(mean(x[r]^2) + eps) * gain, rows of d_model
 * (a multiple of 8); y may alias x.
 */
int pgsr_rmsnorm_bf16(int32_t n, int32_t d_model, const void *x, const void *gain, float eps, void *y,
                      void *stream);
/*
 * Rotary embedding in place on x [n][n_heads][head_dim] (head_dim even): for
 * i < head_dim/2 the pair (x_i, x_{i + head_dim/2}) of token t turns by
 * positions[t] * theta^(-2i/head_dim).  positions: device int32 [n], the
 * tokens' absolute positions, so a replay from P rotates exactly as the full
 * run does.  The angle is reduced in fp64.
 */
int pgsr_rope_bf16(int32_t n, int32_t n_heads, int32_t head_dim, void *x, const int32_t *positions,
                   double theta, void *stream);
/*
 * SwiGLU gate: out[r][j] = SiLU(gate_up[r][j]) * gate_up[r][d_ff + j] with
 * SiLU(g) = g / (1 + e^-g); gate_up [n][2 d_ff], out [n][d_ff], d_ff a
 * multiple of 8.
 */
int pgsr_silu_mul_bf16(int32_t n, int32_t d_ff, const void *gate_up, void *out, void *stream);

/*
 * Next-token sampling for the re-decode of model-derived suffix content
 * (Section 3.2, after Lemma 2), deterministic as Theorem 1's assumption A1
 * asks: the randomness source is fixed by (seed, stream, position).
 * For row i < n of logits [n][vocab] (device, row-major, dtype PGSR_F32 or
 * PGSR_BF16):
 *   temperature > 0: tokens[i] = argmax_v (logits[i][v] / temperature
 *                     - log(-log u)), scores in fp32, where u for entry v is
 *                     word (v mod 4) of Philox4x64-10 (Salmon et al., SC 2011)
 *                     on counter (v div 4, positions[i], streams[i], 0) and
 *                     key (seed, 0), mapped x -> (floor(x / 2^41) + 1/2) / 2^23;
 *   temperature == 0: tokens[i] = argmax_v logits[i][v] (greedy).
 * Ties go to the lowest index; NaN scores never win.  streams, positions: host
 * int64 arrays of n; tokens: device int32 [n].  With a device workspace of at
 * least pgsr_sample_workspace_bytes(n, vocab) bytes the vocabulary is split
 * over several workgroups per row (same result); workspace may be NULL.
 * PGSR_EINVAL on a bad size, pointer or temperature (negative, NaN, inf).
 */
size_t pgsr_sample_workspace_bytes(int32_t n, int32_t vocab);
int pgsr_sample_tokens(int32_t n, int32_t vocab, int32_t dtype, const void *logits, float temperature,
                       uint64_t seed, const int64_t *streams, const int64_t *positions, void *workspace,
                       size_t workspace_bytes, int32_t *tokens, void *stream);

/* ======================================================================== *
 * Forget front-end: the provenance queries and checkpoint selection that turn
 * a forget request for target z into the crop length of the restore
 * (Algorithm 1, the steps before the restore; Section 3.4 (a) and (b);
 * Lemma 2; Corollary 1).  Host code only: no device access, no stream.
 * Handles are not thread-safe; distinct handles may be used concurrently.
 * Calls validate everything before changing anything (all-or-nothing).
 *
 * Readings where the paper is silent:
 *   turns are 1-indexed; a checkpoint boundary b >= 0 names the state after
 *   turn b; artifacts arrive in non-decreasing turn order; a parent must
 *   already exist and belong to the same or an earlier turn (so ids are a
 *   topological order of the DAG); the artifacts where z enters are those
 *   whose own source ids contain z, and all of them seed the closure; the KV
 *   length after turn b is the largest span end over turns <= b; among
 *   checkpoints with equal boundaries the last registered wins.
 * ======================================================================== */

/* Artifact types of the recorded data flow (Section 3.4 (a)). */
enum {
    PGSR_ART_MEMORY_FIELD = 0, PGSR_ART_PROMPT_BLOCK = 1, PGSR_ART_MODEL_TURN = 2,
    PGSR_ART_REPLY = 3, PGSR_ART_PLAN = 4, PGSR_ART_TOOL_CALL = 5,
    PGSR_ART_OBSERVATION = 6, PGSR_ART_SUMMARY = 7
};

/* Checkpoint placement policies (the granularity ablation of Section 4):
 * every turn boundary 0..T-1; the session start only; 0 and the boundary
 * before every turn that introduces a source id; every k-th boundary. */
enum {
    PGSR_POLICY_EVERY_TURN = 0, PGSR_POLICY_SESSION_START = 1,
    PGSR_POLICY_BEFORE_INJECTION = 2, PGSR_POLICY_EVERY_K = 3
};

typedef struct pgsr_graph pgsr_graph;
typedef struct pgsr_ckpt_store pgsr_ckpt_store;

/* Result of a forget query (Algorithm 1: locate the source, first entry
 * boundary, taint closure, restore point c*). */
typedef struct pgsr_forget_plan {
    int64_t tau;                  /* first entry boundary: earliest turn where z entered */
    int64_t checkpoint;           /* index of c* in registration order */
    int64_t boundary;             /* boundary(c*) < tau */
    int64_t crop_len;             /* token offset of c*: the length pgsr_kv_crop keeps */
    int64_t seq;                  /* cache handle (sequence id) of c* */
    int64_t env_snapshot;         /* environment snapshot id of c* */
    int64_t manifest;             /* prompt manifest id of c* */
    int64_t replay_transitions;   /* T - boundary(c*) (Corollary 1) */
    int64_t minimal_transitions;  /* T - tau + 1 (Corollary 1 lower bound) */
    int64_t n_sources;            /* artifacts where z entered */
    int64_t closure_size;         /* |I(z)| (Lemma 2) */
    int64_t clean_artifacts;      /* |{a : turn(a) < tau}| (Lemma 2 (ii)) */
    int64_t committed_after_tau;  /* artifacts of turns >= tau with an external side effect */
} pgsr_forget_plan;

/* Provenance graph G (Section 3.4 (a)) with room for max_artifacts artifacts,
 * max_edges parent references and max_sources source-id references in total;
 * all host memory is reserved here.  PGSR_EINVAL on a negative size. */
int pgsr_graph_create(int64_t max_artifacts, int64_t max_edges, int64_t max_sources,
                      pgsr_graph **out);
/* NULL is a no-op. */
int pgsr_graph_destroy(pgsr_graph *g);

/*
 * Record n artifacts (ids size .. size+n-1, in order; Lemma 2 (i): G only
 * grows).  Host arrays of length n: types (PGSR_ART_*), turns (>= 1, not
 * decreasing, including against the last recorded artifact), span_begin /
 * span_end (0 <= begin <= end, tokens of the KV timeline), committed (0/1,
 * may be NULL = none).  Parents of artifact i are parents[parent_off[i] ..
 * parent_off[i+1]) (parent_off has n+1 entries, starting at 0, not
 * decreasing); each is an existing id or an earlier one of this batch, of a
 * turn <= turn[i].  Source ids it introduces: sources[source_off[i] ..
 * source_off[i+1]), same convention.  parents / sources may be NULL when the
 * offsets are all 0.  *first_id (may be NULL) receives the first new id.
 * PGSR_EINVAL on a bad record, PGSR_ENOMEM past the capacity; then nothing is
 * recorded.
 */
int pgsr_graph_append(pgsr_graph *g, int64_t n, const int32_t *types, const int32_t *turns,
                      const int64_t *span_begin, const int64_t *span_end,
                      const int64_t *parent_off, const int64_t *parents,
                      const int64_t *source_off, const int64_t *sources,
                      const uint8_t *committed, int64_t *first_id);

/* Artifacts recorded; T (the last turn, 0 when empty); tokens in the cache
 * once turn b is done (b >= 0). */
int pgsr_graph_size(const pgsr_graph *g, int64_t *n_out);
int pgsr_graph_session_length(const pgsr_graph *g, int64_t *T_out);
int pgsr_graph_kv_length_after(const pgsr_graph *g, int64_t b, int64_t *len_out);

/* Locate the source (Algorithm 1): ids of the artifacts where z entered, in
 * ascending order, into out[0 .. capacity); *n_out = their number.  Returns
 * PGSR_ERANGE (writing nothing) when capacity is too small; out may be NULL
 * with capacity 0 to ask for the count. */
int pgsr_graph_locate_source(const pgsr_graph *g, int64_t z, int64_t *out, int64_t capacity,
                             int64_t *n_out);

/* Taint closure (Lemma 2): the seeds and every artifact reachable from them,
 * ascending ids, same output convention as pgsr_graph_locate_source.  Seeds
 * must be existing ids. */
int pgsr_graph_taint_closure(const pgsr_graph *g, const int64_t *seeds, int64_t n_seeds,
                             int64_t *out, int64_t capacity, int64_t *n_out);

/* Boundaries a placement policy yields for the recorded session, ascending,
 * same output convention; k >= 1 for PGSR_POLICY_EVERY_K (ignored otherwise). */
int pgsr_graph_policy_boundaries(const pgsr_graph *g, int32_t policy, int64_t k, int64_t *out,
                                 int64_t capacity, int64_t *n_out);

/* Checkpoint set C (Section 3.4 (b)): metadata only -- the boundary, the token
 * offset the restore crops to, the cache handle, environment snapshot and
 * prompt manifest ids; no tensor copies (40 bytes per checkpoint). */
int pgsr_ckpt_create(int64_t capacity, pgsr_ckpt_store **out);
int pgsr_ckpt_destroy(pgsr_ckpt_store *s);
/* PGSR_EINVAL on a negative boundary or offset, PGSR_ENOMEM when full. */
int pgsr_ckpt_register(pgsr_ckpt_store *s, int64_t boundary, int64_t token_offset, int64_t seq,
                       int64_t env_snapshot, int64_t manifest);
int pgsr_ckpt_count(const pgsr_ckpt_store *s, int64_t *n_out);

/*
 * The forget query of Algorithm 1 for target z: locate where z entered, its
 * first entry boundary tau, the taint closure I(z), and the restore point
 * c* = argmax {c : boundary(c) < tau}.  Fills *plan; when closure is not NULL
 * also writes I(z) (ascending ids) into closure[0 .. capacity).
 * PGSR_ENOENT when z never entered or no checkpoint lies below tau;
 * PGSR_ERANGE when capacity < |I(z)| (plan->closure_size is still set, the
 * closure buffer untouched).  The restore is then pgsr_kv_crop of sequence
 * plan->seq to plan->crop_len tokens (as int32) on the pool that holds it.
 */
int pgsr_forget_plan_query(const pgsr_graph *g, const pgsr_ckpt_store *s, int64_t z,
                           int64_t *closure, int64_t capacity, pgsr_forget_plan *plan);

#ifdef __cplusplus
}
#endif

#endif /* PGSR_H */
