/*
 * fademem.h -- C ABI of the FadeMem per-chunk cache step on one MI355X
 * (gfx950).  FadeMem: "Distance-Aware Memory Consolidation for
 * Autoregressive Video Diffusion", arXiv 2606.10671.
 *
 * The library keeps, per transformer layer, the bounded ordered memory of
 * Sec. 3.1 / Sec. 3.3 (at most M entries, each one representative KV block
 * plus its span s and temporal position mu), updates it with Algorithm S1
 * (append, power-law distance schedule, adjacent-pair consolidation,
 * first-frame anchor), and runs the attention of a chunk's queries over
 * [memory entries in order || current chunk] (Sec. 3.1, Sec. 4.1).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Tensors are token-major and contiguous: a block, a query chunk, a
 *   current chunk and an output are [tokens][heads][head_dim], one batch.
 *   Element type is fp32 or bf16 as configured (dtype); LSE is fp32.
 * - Device pointers must be 16-byte aligned; the pool 256-byte aligned.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   Every call except fademem_get_state, fademem_entry_kv, fademem_set_state,
 *   fademem_merge_log, fademem_merge_counts and fademem_verify is
 *   asynchronous on that stream and never waits for the device
 *   (fademem_stage and fademem_count only read host state).  One cache is
 *   used by one host thread and one stream at a time.
 * - Calls that implement a step of the method cite the passage that defines
 *   it; the plumbing around them (pool sizing, creation, readers,
 *   checkpointing, error strings) has no counterpart in the paper and cites
 *   none.
 * - Ownership: the caller allocates and owns the device pool and every
 *   Q/K/V/O/LSE buffer.  The library allocates no device memory, never
 *   frees caller memory and keeps only the pool pointer.  insert copies K
 *   and V, so the caller may reuse its buffers once the stream has passed
 *   the call.
 * - Errors: 0 (FADEMEM_OK) or a negative FADEMEM_E* code.  Arguments and
 *   state are validated before anything is enqueued, so a call that fails
 *   validation leaves the cache unchanged.  FADEMEM_EHIP reports a HIP
 *   launch or runtime failure (see fademem_last_hip_error).  No C++
 *   exception crosses this interface.
 * - Debugging: with the environment variable FADEMEM_SERIALIZE set (not
 *   "0") when a cache is created, every asynchronous call on it waits for
 *   its own work before returning and reports a failure of that work as
 *   FADEMEM_EHIP, so an error shows at the call that caused it.  Results
 *   are the same bits as without it.
 */
#ifndef FADEMEM_H
#define FADEMEM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  FADEMEM_OK = 0,
  FADEMEM_EINVAL = -1,     /* bad configuration, argument, pointer or size      */
  FADEMEM_ESTATE = -2,     /* call not allowed in the current memory state       */
  FADEMEM_ENOMEM = -3,     /* caller's pool smaller than fademem_pool_bytes      */
  FADEMEM_EHIP = -4,       /* HIP runtime or launch error                        */
  FADEMEM_EUNSUPPORTED = -5,/* valid request this build does not implement       */
  FADEMEM_EINTERNAL = -6,  /* host replay of the memory state disagrees with the
                              device (fademem_verify, serialize mode)           */
  FADEMEM_ESCRATCH = -7    /* request larger than the static scratch of an
                              allocation-free entry point                       */
};

enum { FADEMEM_F32 = 0, FADEMEM_BF16 = 1 };

/* Consolidation operators: the K, V rule of a merge (Sec. 3.3
 * "Consolidation operator"; the ablation of Sec. 4.3, Table 4).  The
 * metadata rule (spans add, mu span-weighted) and the anchor's branch are
 * the same for all.
 *   SQRT_SPAN      X = (sqrt(s_j) X_j + sqrt(s_j+1) X_j+1) / (sqrt(s_j) + sqrt(s_j+1)),
 *                  the paper's default, in fp64, one RNE rounding to the storage type;
 *   AVERAGE        the same with both weights 1/2 (unweighted average);
 *   SELECT_NEAREST the newer entry's K, V (representative selection; no
 *                  K/V bytes move: the merged entry takes the newer one's slot);
 *   MAX            elementwise max pooling; the newer value wins only when
 *                  strictly greater (equal values, -0 and +0 included, keep
 *                  the older entry's bits). */
enum {
  FADEMEM_MERGE_SQRT_SPAN = 0,
  FADEMEM_MERGE_AVERAGE = 1,
  FADEMEM_MERGE_SELECT_NEAREST = 2,
  FADEMEM_MERGE_MAX = 3
};

typedef struct fademem_config {
  int64_t budget;           /* M, the entry budget (Sec. 3.1); 2 <= M <= 1023.
                               M >= 2 keeps one pair eligible once the newest
                               entry is protected (Sec. 3.3).                  */
  int32_t heads;            /* H >= 1                                          */
  int32_t head_dim;         /* D, 64 or 128                                    */
  int64_t tokens_per_block; /* N >= 1, tokens of one generation unit (one
                               latent frame, supplementary Sec. S4)            */
  double beta;              /* exponent of u(d) = d^beta, 0 < beta <= 1
                               (Sec. 3.3); the paper's default is 0.3 (Sec. 4.1) */
  int32_t anchor;           /* 1: the first inserted block is a global anchor
                               (Sec. 3.3, Alg. S1), the paper's default; 0: off */
  int32_t merge_op;         /* FADEMEM_MERGE_* (default SQRT_SPAN)              */
  int32_t dtype;            /* FADEMEM_F32 or FADEMEM_BF16 for K, V, Q, O      */
  int32_t layers;           /* L >= 1 per-layer memories sharing one schedule.
                               The schedule depends only on positions, so every
                               layer makes the same decisions (Sec. 3.3).       */
  int32_t rope_pairs;       /* Temporal RoPE handling (Sec. 3.3 "Boundary and
                               positional handling"): 0 = off (keys are used as
                               stored).  P > 0: the first P interleaved pairs
                               (2i, 2i+1) of each head's dimension carry the
                               temporal rotary phase; 1 <= P <= D/2.  Blocks
                               are inserted without their temporal phase and
                               stored so; fademem_attend exposes memory entry
                               i (0 = oldest) at temporal index i, i.e. pair k
                               of its keys rotated by the angle i * w_k with
                               w_k = rope_theta^(-k/P), evaluated in fp64 and
                               rounded once to the storage type.  The caller
                               applies the same rotation to the current
                               chunk's queries and keys at indices n + f (n =
                               entries held, f = frame within the chunk).    */
  double  rope_theta;       /* rotary base (> 1), e.g. 10000; ignored if P = 0 */
  int32_t stage_frames;     /* 0..4: frames a chunk may stage for the
                               zero-copy update (fademem_stage); 0 = off.
                               The pool then holds M + max(1, stage_frames)
                               KV slots per layer.                            */
} fademem_config;

typedef struct fademem_cache fademem_cache; /* opaque host object */

/* Bytes of device pool a configuration needs: M + max(1, stage_frames) KV
 * slots per layer for K and V, the memory's metadata, the attention's
 * scratch for split work (bf16: partial results of split query tiles,
 * 70.3 MB at D = 128; fp32: partial results of key ranges, 512 x 64 x (D+2)
 * floats) and, with rope_pairs > 0, a re-indexed K view per layer (one K
 * block per slot).  Returns EINVAL for a bad config. */
int fademem_pool_bytes(const fademem_config* cfg, size_t* bytes);

/* Create a cache over a caller-owned device pool of `pool_bytes` bytes
 * (>= fademem_pool_bytes).  Enqueues the initialisation of the metadata on
 * `stream` (the pool's previous contents do not matter).  The memory starts
 * empty.  *out receives a host handle to destroy with fademem_cache_destroy.
 * Errors: EINVAL (config, NULL or misaligned pool), ENOMEM (pool too small),
 * EHIP. */
int fademem_cache_create(const fademem_config* cfg, void* dev_pool, size_t pool_bytes,
                         void* stream, fademem_cache** out);

/* Release the host handle.  The pool stays the caller's.  NULL is a no-op. */
int fademem_cache_destroy(fademem_cache* cache);

/* Append the block B_t = (K_t, V_t) at position t as the entry (K_t, V_t,
 * t, 1) -- first step of Alg. S1, Sec. 3.3 "Memory entries and insertion".
 * k[l], v[l] (host arrays of `layers` device pointers) are layer l's block,
 * [N][H][D].  Positions are integers that strictly increase (0-indexed by
 * convention; the first block inserted into an empty memory becomes the
 * anchor when the option is on), |t| < 2^40.
 * Errors: EINVAL (NULL/misaligned pointers, position out of range),
 * ESTATE (position not increasing, or M+1 entries already held: call
 * fademem_consolidate first), EHIP. */
int fademem_insert(fademem_cache* cache, const void* const* k, const void* const* v,
                   int64_t position, void* stream);

/* Rest of Alg. S1.  If the memory holds at most M entries this is a no-op
 * (and enqueues nothing).  Otherwise, on the device: d_i = t - mu_i with t
 * the newest position, u = d^beta, gaps |u(d_{i+1}) - u(d_i)| over the
 * adjacent pairs except the one holding the newest entry, j = the smallest
 * gap (gaps within a relative 1e-9 of the smallest count as tied and the
 * oldest such pair wins); the pair is replaced by its consolidation: spans
 * add, mu is span-weighted; K, V by the configured operator (default:
 * sqrt-span weighted average evaluated in fp64 and rounded once,
 * round-to-nearest-even, to the storage type); when the pair holds the
 * anchor its K, V and position are kept (Sec. 3.3, Alg. S1).  The decision
 * never crosses to the host.  Errors: EHIP. */
int fademem_consolidate(fademem_cache* cache, void* stream);

/* A chunk's F updates in one call: for f = 0..frames-1, append frame f at
 * position first_position + f, then consolidate when over budget -- the
 * F sequential Alg. S1 updates that follow a chunk's final denoising step
 * (Sec. 4.1; supplementary Sec. S4: one entry per latent frame).  State,
 * merge log and every stored K/V bit equal those of `frames` calls of
 * fademem_insert + fademem_consolidate.  Frames are taken in groups of up
 * to four; within a group each K/V block that changes is written once (a
 * chain of merges is evaluated in registers, each merge
 * rounded to the storage type as on its own), and frames that a merge of
 * the same call consumes are read from the caller's buffers, never copied
 * into the pool.  k[l], v[l] (host arrays of `layers` device pointers) are
 * layer l's chunk, [frames*N][H][D], frame f in rows f*N..(f+1)*N-1; the
 * caller may reuse them once the stream has passed the call.
 * Errors: EINVAL (NULL/misaligned pointers, frames < 1, positions out of
 * range), ESTATE (first_position not above the newest position, or M+1
 * entries held), EHIP. */
int fademem_update(fademem_cache* cache, const void* const* k, const void* const* v, int64_t frames,
                   int64_t first_position, void* stream);

/* Zero-copy insert (Alg. S1 "Append"; Sec. 4.1 and supplementary Sec. S4:
 * one entry per latent frame, the memory updated once the chunk is
 * generated).  With stage_frames > 0, the caller's projection can write a
 * chunk's K/V straight into free pool slots instead of its own buffers:
 * fademem_stage returns, for frame f < frames of layer l, the device
 * address of the K block k[l*frames + f] and of the V block
 * v[l*frames + f] ([N][H][D] each; the frames of a chunk are separate
 * blocks).  It reads host state only and enqueues nothing; the addresses
 * stay valid until the next insert, consolidate or update.
 * fademem_update_staged(frames, first_position) then runs the same F
 * Alg. S1 updates as fademem_update with frame f taken from its staging
 * slot: a frame that survives stays where the caller wrote it (no copy) and
 * one that a merge consumes frees its slot.  State, merge log and stored
 * K/V bits equal those of fademem_update on the same frames.
 * fademem_attend_staged attends over [memory || staged frames] (the
 * generator's final pass over a chunk, whose K/V become the update's).
 * The free slots are known on the host because the library replays every
 * update's schedule on the host copy of the integer metadata (the device
 * still makes the decisions; fademem_verify checks that both agree).
 * Limits: 1 <= frames <= stage_frames <= 4.  Errors: EINVAL (frames out of
 * range, NULL pointers, positions out of range), ESTATE (M+1 entries held,
 * position not above the newest), EHIP. */
int fademem_stage(fademem_cache* cache, int64_t frames, void** k, void** v);
int fademem_update_staged(fademem_cache* cache, int64_t frames, int64_t first_position, void* stream);
int fademem_attend_staged(fademem_cache* cache, int32_t layer, const void* q, int64_t q_tokens,
                          int64_t frames, float scale, void* out, float* lse, void* stream);

/* Attention of the chunk's queries over layer `layer`'s exposed cache:
 * O_h = softmax(scale * Q_h K_h^T) V_h per head, with the keys/values
 * [memory entries in memory order || current chunk] (Sec. 3.1, Sec. 4.1),
 * no mask.  q and out: [q_tokens][H][D]; k_cur, v_cur: [cur_tokens][H][D]
 * (cur_tokens may be 0 if the memory is not empty).  scale = 0 selects
 * 1/sqrt(D).  lse, if not NULL, receives [H][q_tokens] fp32 natural-log
 * sums of exponentials of the scaled scores.  Accumulation is fp32 (bf16
 * inputs use bf16 MFMA with fp32 accumulation).  q_tokens = 0 is a no-op.
 * Errors: EINVAL (layer out of range, NULL/misaligned pointers, no keys at
 * all, sizes out of range), EHIP. */
int fademem_attend(fademem_cache* cache, int32_t layer, const void* q, int64_t q_tokens,
                   const void* k_cur, const void* v_cur, int64_t cur_tokens, float scale,
                   void* out, float* lse, void* stream);

/* Number of entries currently held (host mirror; never waits). */
int fademem_count(const fademem_cache* cache, int64_t* count);

/* Copy the memory's metadata to host arrays of at least M+1 elements (any
 * of them may be NULL): first covered position, span s_i, pos_sum_i (the
 * integer with mu_i = pos_sum_i / s_i) and the newest position.
 * Synchronises `stream`.  Errors: EINVAL, EHIP. */
int fademem_get_state(fademem_cache* cache, int64_t* count, int64_t* first, int64_t* span,
                      int64_t* pos_sum, int64_t* newest, void* stream);

/* Device pointers of layer `layer`'s logical entry i (0 = oldest), valid
 * until the next insert/consolidate.  Synchronises `stream`. */
int fademem_entry_kv(fademem_cache* cache, int32_t layer, int64_t i, const void** k,
                     const void** v, void* stream);

/* Checkpoint / resume: put a saved memory into a cache that holds nothing
 * yet (just created, same configuration), so that it continues exactly as
 * the cache the state was saved from.  count (0..M) entries, oldest first:
 * first[i], span[i], pos_sum[i] as fademem_get_state returns them, and the
 * newest inserted position; k[l*count + i], v[l*count + i] (host arrays of
 * layers*count device pointers, [N][H][D] each) are entry i's K, V of layer
 * l, e.g. from fademem_entry_kv of the saved cache or the caller's copies of
 * them (the saved state holds nothing else: entry 0 is the anchor when the
 * option is on).  The merge log and counts start again from zero.  Copies
 * on `stream` and synchronises it.  Errors: EINVAL (NULL/misaligned
 * pointers, count > M, spans < 1, first not increasing by at least the
 * previous span, pos_sum outside [first*span, newest*span], newest below
 * the last covered position, positions out of range), ESTATE (the cache
 * already holds or has held entries), EHIP. */
int fademem_set_state(fademem_cache* cache, int64_t count, const int64_t* first, const int64_t* span,
                      const int64_t* pos_sum, int64_t newest, const void* const* k, const void* const* v,
                      void* stream);

/* Selected pair indices j of the consolidations run so far, oldest first.
 * *total receives how many have run; the most recent min(total, cap, 4096)
 * are copied into j[].  Synchronises `stream`. */
int fademem_merge_log(fademem_cache* cache, int32_t* j, int64_t cap, int64_t* total,
                      void* stream);

/* Counts of the consolidations run so far (Algorithm S1's merge step):
 * *total of them, *anchor of which merged the anchor's pair (no K/V work),
 * so total - anchor merges moved K/V bytes.  Either pointer may be NULL.
 * Unlike the log these counts are not capped.  Synchronises `stream`.
 * Errors: EINVAL (NULL cache), EHIP. */
int fademem_merge_counts(fademem_cache* cache, int64_t* total, int64_t* anchor, void* stream);

/* Distance-dependent spectral decay (Sec. 3.2; supplementary Sec. S2).
 * latents: device [clips][frames][height][width] fp32, channel-averaged
 * latent frames.  For every clip the orthonormal 2-D DCT-II of frames
 * 0..max_lag; for every radial band k < bands and lag the Pearson
 * correlation of band k's DCT coefficients of frame 0 and of frame lag;
 * corr (device, [bands][max_lag+1] fp64) receives the mean over clips.
 * band_of: device [height][width] int32, the band of DCT coefficient
 * (u, v) (any value outside [0, bands) leaves the coefficient out).
 * workspace: device, 256-byte aligned, at least
 * fademem_spectral_workspace_bytes (the DCT bases, the band order and the
 * per-clip band sums; frames of up to 64 x 128 are transformed on chip,
 * larger ones also keep the DCT of the analysed frames there).  Limits:
 * height*width <= 40960 and, above 64 x 128, the frame, its transform and
 * both DCT bases within 160 KiB of LDS; max_lag < frames, max_lag < 65535;
 * 1 <= bands <= 1024.  Asynchronous on `stream`; the library allocates
 * nothing.  Every call with the same inputs gives the same bits.  A band
 * whose coefficients do not vary, or that holds none, gets NaN.
 * Errors: EINVAL (NULL/misaligned pointers, sizes out of range), ENOMEM
 * (workspace too small), EHIP. */
int fademem_spectral_workspace_bytes(int64_t clips, int64_t frames, int32_t height, int32_t width,
                                     int32_t bands, int64_t max_lag, size_t* bytes);
int fademem_spectral_corr(const float* latents, int64_t clips, int64_t frames, int32_t height,
                          int32_t width, const int32_t* band_of, int32_t bands, int64_t max_lag,
                          void* workspace, size_t workspace_bytes, double* corr, void* stream);

/* Synchronise `stream` and compare the host replay of the memory (spans,
 * positions, slot table) with the device's state.  Returns OK or
 * EINTERNAL (serialize mode runs the same check after every call).
 * Errors: EINVAL (NULL cache), EHIP. */
int fademem_verify(fademem_cache* cache, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * analysis as fademem_spectral_corr, with its workspace in a static scratch
 * array of the library (64 MiB per GPU, held by each GPU the library runs on
 * until the process ends) instead of a caller's buffer; the caller still
 * passes the inputs and corr.  The call allocates nothing.  Requests whose
 * workspace (fademem_spectral_workspace_bytes) exceeds 64 MiB return
 * FADEMEM_ESCRATCH before anything is enqueued (the 374-clip analysis of
 * supplementary Sec. S2 needs 38.2 MB).  All calls on one GPU share its
 * scratch: calls that overlap on one GPU (several streams or threads) race.
 * Errors: as fademem_spectral_corr, plus ESCRATCH. */
int fademem_spectral_corr_static(const float* latents, int64_t clips, int64_t frames, int32_t height,
                                 int32_t width, const int32_t* band_of, int32_t bands, int64_t max_lag,
                                 double* corr, void* stream);

/* Host steps of the spectral-decay analysis (Sec. 3.2; supplementary Sec.
 * S2) on small host arrays; they read and write host memory only, enqueue
 * nothing and need no device.  The paper gives the radial frequency, the
 * horizon as the onset of the near-flat regime after the main decay, and a
 * nonlinear least-squares fit of r*(t) = a t^(-b); the band edges, the
 * smoothing and the threshold are this library's readings.
 *
 * fademem_spectral_band_map: band_of (host int32 [height][width]) receives
 * the band of DCT coefficient (u, v): `bands` equal-width bins of
 * r = sqrt((u/H)^2 + (v/W)^2) over [0, max r], the last bin closed, the DC
 * coefficient -1 (left out); centres (host double [bands], may be NULL)
 * the bins' centre radii.  1 <= height, width <= 1024, 1 <= bands <= 1024.
 *
 * fademem_spectral_horizons: corr (host double [bands][lags], row k = band
 * k's C_k(lag)); each row is smoothed by a centred moving average over
 * `window` lags (shrinking at the ends); horizon[k] (host int64 [bands]) is
 * the first lag >= 1 at which the smoothed curve has made at least half of
 * its total decay and falls to the next lag by less than `drop` times its
 * steepest one-lag fall, or -1 (the defaults used here: window 5, drop 0.05).
 *
 * fademem_spectral_fit: (a, b) of r = a t^(-b) minimising sum (r_i - a
 * t_i^(-b))^2 over n >= 2 points with t_i, r_i > 0: Gauss-Newton from the
 * straight-line fit of log r on log t, at most `iters` steps.
 *
 * Errors: EINVAL (NULL pointers, sizes out of range, non-positive or
 * infinite points, a fit that does not converge to finite values), ENOMEM. */
int fademem_spectral_band_map(int32_t height, int32_t width, int32_t bands, int32_t* band_of, double* centres);
int fademem_spectral_horizons(const double* corr, int32_t bands, int64_t lags, int32_t window, double drop,
                              int64_t* horizon);
int fademem_spectral_fit(const double* t, const double* r, int64_t n, int32_t iters, double* a, double* b);

/* hipError_t value of the last FADEMEM_EHIP on this cache (0 if none). */
int fademem_last_hip_error(const fademem_cache* cache);

/* Static description of an error code. */
const char* fademem_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* FADEMEM_H */
