/*
 * libprotokv -- ProtoKV far-memory hot path on one AMD Instinct MI355X (gfx950).
 *
 * ProtoKV keeps, per (layer, KV head), an exact near window of the last W
 * frames' KV and a fixed-capacity bank of K prototypes that absorbs every
 * token evicted from that window (paper: Section "State representation and
 * prototype bank", Section "Online update: eviction, assignment, and
 * prototype maintenance", Appendix Algorithm "ProtoKV Streaming Update").
 * At query time each active prototype is exposed as S pseudo-tokens decoded
 * from its PQ residual histograms (Section "Residual Statistics and
 * Pseudo-Token Interface", Algorithms "DecodeTopSResidualModes" and
 * "Pseudo-Token Decoding and Attention") and attention runs over
 * [near KV ; pseudo-tokens] with the log-mass logit bias of Eq. attn_logit.
 *
 * Calling conventions (every entry point):
 *  - All arguments are plain pointers and sizes.  "device" pointers are HIP
 *    device memory of the current device; "host" pointers are ordinary host
 *    memory.  `stream` is a hipStream_t passed as void* (NULL = the default
 *    stream); work is enqueued on it and the call returns without waiting,
 *    unless the description says the call synchronizes.
 *  - The caller owns all device memory, including the workspace; the
 *    library never allocates device memory.  Input pointers are borrowed
 *    until the enqueued work has completed on `stream`.
 *  - A handle is not thread-safe; calls on one handle must be serialized.
 *  - Every function returns a protokv_status.  Argument and state checks are
 *    done on the host before anything is enqueued, so a non-OK return leaves
 *    the handle and the device untouched, except PROTOKV_E_DEVICE, which
 *    reports a HIP error from a launch or copy.  protokv_last_error() gives a
 *    human-readable message for the last failure on a handle.
 *
 * v1 supports head_dim = 128, G = 8 PQ subspaces of 16 dims, C <= 16
 * codewords, S <= 16 pseudo-tokens per prototype and smoothing eps = 1.
 */
#ifndef PROTOKV_H
#define PROTOKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct protokv_ctx* protokv_t;

typedef enum {
  PROTOKV_OK = 0,
  PROTOKV_E_INVALID = 1,     /* malformed argument or configuration */
  PROTOKV_E_UNSUPPORTED = 2, /* well-formed but outside what v1 implements */
  PROTOKV_E_WORKSPACE = 3,   /* workspace missing, too small or misaligned */
  PROTOKV_E_STATE = 4,       /* call out of order for the stream's state */
  PROTOKV_E_DEVICE = 5       /* HIP runtime error */
} protokv_status;

enum { PROTOKV_KV_BF16 = 0, PROTOKV_KV_FP32 = 1 };

/* flags */
enum {
  PROTOKV_FLAG_PQ = 1u,        /* residual statistics on (off = "w/o residual stats" ablation) */
  PROTOKV_FLAG_MASS_BIAS = 2u, /* log-mass bias on (off = "b_k = 0" ablation) */
  PROTOKV_FLAG_MAINTENANCE = 4u, /* Alg. "Prototype Maintenance" after every fold (capacity <= 2048) */
  PROTOKV_FLAG_EMA_CENTRES = 8u, /* Alg. "ProtoKV Streaming Update" fixed-rate EMA centres (not with maintenance) */
  PROTOKV_FLAG_MAH_SQUARED = 16u, /* Eq. 1's spatial term as the squared Mahalanobis distance d^T (Sigma + rho I)^-1 d
                                    (default: its square root, the distance) */
  PROTOKV_FLAG_VAR_ALLOC = 32u    /* appendix "Dynamic Pseudo-Token Allocation": S_k pseudo-tokens per prototype
                                     in proportion to its residual variance (capacity <= 4096); see
                                     protokv_synthesize */
};

typedef struct {
  int32_t num_streams;      /* independent streams sharing one workspace */
  int32_t num_layers;       /* L */
  int32_t num_kv_heads;     /* Hkv */
  int32_t num_q_heads;      /* Hq, a multiple of Hkv (GQA) */
  int32_t head_dim;         /* D, must be 128 */
  int32_t grid_h, grid_w;   /* visual tokens per frame T = grid_h * grid_w, raster order */
  int32_t window_frames;    /* near window W in frames (W * T tokens) */
  int32_t capacity;         /* K_max prototype slots per (stream, layer, kv head), 1..65535 */
  int32_t pseudo_per_proto; /* S */
  int32_t pq_subspaces;     /* G, must be 8 */
  int32_t pq_codewords;     /* C, 2..16 */
  int32_t beam;             /* B >= S; the decoded top-S does not depend on B (exact beam) */
  int32_t t_idle;           /* T_idle in frames */
  int32_t max_query_tokens; /* largest Tq passed to protokv_attend */
  int32_t kv_dtype;         /* PROTOKV_KV_BF16 or PROTOKV_KV_FP32 */
  uint32_t flags;           /* PROTOKV_FLAG_* */
  float eta;                /* spatial EMA rate */
  float pq_eps;             /* PQ smoothing, must be 1 */
  double lambda_sp;         /* spatial weight of Eq. 1 */
  double lambda_idle;       /* idle weight of Eq. 1 */
  double ridge;             /* rho added to Sigma's diagonal in d_Mah */
  double gamma;             /* maintenance: idle mass decay, n <- floor((1 - gamma) n), in [0, 1) */
  double eps_k, eps_v;      /* maintenance: key / value centre merge thresholds (>= 0) */
  float alpha, beta;        /* PROTOKV_FLAG_EMA_CENTRES: key / value centre EMA rates, in [0, 1] */
  double rope_theta;        /* rotary positions in the readout: 0 = off, else the base (> 1) */
  int32_t warm_frames;      /* codebook warm-up folds T_warm (0 = use the given codebooks throughout) */
  int32_t warm_tokens;      /* warm-up reservoir capacity per (stream, layer, kv head), 1..65536 */
  int32_t kmeans_epochs;    /* mini-batch k-means passes over the reservoir, >= 1 */
  int32_t kmeans_batch;     /* mini-batch size, 1..64 */
  int32_t pseudo_max;       /* PROTOKV_FLAG_VAR_ALLOC: largest S_k, pseudo_per_proto..16 */
} protokv_config;

/* Table tab:default_config defaults (S=8, lambda_sp=0.1, lambda_idle=0.01,
 * T_idle=120, eta=0.05, alpha=beta=0.05, G=8, C=16, B=32, gamma=0.05,
 * eps_K=0.20, eps_V=0.25; maintenance, EMA centres, RoPE and the codebook
 * warm-up off, warm_tokens=1024, kmeans_epochs=4, kmeans_batch=64; variance-aware
 * allocation off, pseudo_max=16) with the 7B-class shape of one
 * stream: 28 layers, 4 KV heads, 28 query heads, 14x14 tokens per frame,
 * W=8 frames, K=256, bf16 KV, PQ and mass bias on, eps=1, rho=1e-4.
 * Host only. */
protokv_status protokv_default_config(protokv_config* cfg);

/* Checks a configuration.  Host only, touches no device. */
protokv_status protokv_validate_config(const protokv_config* cfg);

/* Bytes of device workspace protokv_init needs for `cfg`.  Host only. */
protokv_status protokv_workspace_size(const protokv_config* cfg, size_t* bytes);

/* Creates a handle on the current HIP device.
 * codebooks: host, float32 [num_streams][num_layers][num_kv_heads][2][G][C][D/G]
 *   (index 0 = key codebooks C^K_g, 1 = value codebooks C^V_g; codewords of
 *   subspace g cover dims [g*D/G, (g+1)*D/G)); copied during the call.
 * workspace: device, >= protokv_workspace_size bytes, 256-byte aligned; owned
 *   by the caller, must outlive the handle and must not be touched by the
 *   caller while the handle exists.  It is cleared (empty rings and banks)
 *   on `stream`.
 * Synchronizes `stream` before returning. */
protokv_status protokv_init(const protokv_config* cfg, const float* codebooks,
                            void* workspace, size_t workspace_bytes, void* stream,
                            protokv_t* out);

/* Frees the host handle (not the workspace).  Does not synchronize. */
protokv_status protokv_destroy(protokv_t h);

/* Appends one frame to each listed stream's near window (Alg. "ProtoKV
 * Streaming Update": append to B_near, and once more than W frames are held,
 * mark the oldest frame as evicted; the eviction is absorbed by the next
 * protokv_fold).
 * stream_ids: host, n distinct stream indices.
 * k, v: device, [n][num_layers][num_kv_heads][T][D] in kv_dtype (bf16 or
 *   float32), row-major; entry i belongs to stream_ids[i].  Keys are
 *   unrotated; with rope_theta > 0 a copy rotated at each token's stream
 *   position f * T + j (f = the frame's index in its stream) is kept for
 *   the readout (the fold uses the unrotated keys).
 * Errors: PROTOKV_E_STATE if a listed stream still has an unfolded eviction. */
protokv_status protokv_append_frame(protokv_t h, const int32_t* stream_ids, int32_t n,
                                    const void* k, const void* v, void* stream);

/* Absorbs every pending evicted frame into its stream's prototype bank:
 * seeds free slots (Initialization), assigns the other tokens by Eq. 1 against
 * the post-seed bank and accumulates mass, sum, sum of squares, PQ residual
 * histograms, spatial mean/covariance and recency in eviction order.  With
 * PROTOKV_FLAG_MAINTENANCE each fold then runs Alg. "Prototype Maintenance"
 * on the seeded slots: idle mass decay n <- floor((1 - gamma) n) (sums and
 * squared sums scaled to keep the centre), merging of slot pairs whose key
 * and value centres are closer than eps_k, eps_v (the lower slot absorbs the
 * higher, pairs in ascending order, each merge moving the absorbing centre),
 * and reseeding of emptied slots from the near window's newest tokens.
 * With PROTOKV_FLAG_EMA_CENTRES the centres follow the fixed-rate EMA of
 * Alg. "ProtoKV Streaming Update" instead of running means: the bank's key
 * and value sum fields hold the centres c, p; each absorbed token, in
 * eviction order, sets c <- (1 - alpha) c + alpha K and p <- (1 - beta) p +
 * beta V in float32 (one rounding per product and per add, 1 - alpha
 * rounded first), then its PQ residual codes are taken against the updated
 * centres (the screen's cosine is unchanged; synthesis uses c, p directly).
 * With warm_frames > 0 (appendix "PQ codebook initialization") the first
 * warm_frames folds of a stream count no PQ codes; they append each
 * non-seed token's key and value residuals against its slot's centre
 * sum / n before the fold, in eviction order, to a reservoir of at most
 * warm_tokens per (layer, kv head).  After the last of them, mini-batch
 * k-means learns each subspace's key and value codebook from the
 * reservoir (centres started from rows i * floor(N / C); batches of
 * kmeans_batch consecutive rows assigned with the float32 sequential PQ
 * distance as each batch starts, then each row in order: count += 1,
 * eta = 1 / count, c <- (1 - eta) c + eta x in float32; kmeans_epochs
 * passes), replacing the stream's codebooks from the next fold on (with
 * fewer than C residuals the given codebooks stay).
 * Invalidates any synthesis.  No-op when nothing is pending. */
protokv_status protokv_fold(protokv_t h, void* stream);

/* Decodes the pseudo-tokens of every (layer, kv head) of `stream_id` into the
 * workspace's synthesis buffer (one stream at a time): S pseudo-tokens per
 * active prototype, keys c_k + r^K_s and values p_k + r^V_s rounded to
 * kv_dtype, bias log n_k (Algorithms "DecodeTopSResidualModes" and
 * "Pseudo-Token Decoding and Attention").  The buffer holds the top-S code
 * tuples, the biases and the rows themselves, except for bf16 KV with S >= 5:
 * there it holds no rows, and protokv_attend forms each row from the bank's
 * sums (the centre sum / n, IEEE division) and the code tuples, with the
 * same rounding, as it reads it.  With
 * rope_theta > 0 (Sec. 3.3: the S pseudo-tokens of prototype k share the
 * rotary position tau_k) each pseudo-key, rounded to kv_dtype, is rotated at
 * tau_k in float32 (angle reduced in float64) and rounded again: written
 * that way when the rows are written, turned that way inside protokv_attend
 * when it forms them (the same values either way). */
protokv_status protokv_synthesize(protokv_t h, int32_t stream_id, void* stream);
/* With PROTOKV_FLAG_VAR_ALLOC (appendix "Dynamic Pseudo-Token Allocation")
 * prototype k of each (layer, kv head) is exposed as S_k pseudo-tokens, its
 * top-S_k code tuples (all with bias log n_k), in place of S: the A active
 * prototypes keep the total A * S; each keeps one and the other A * (S - 1)
 * are shared in proportion to Var(H_k), at most pseudo_max each (the excess
 * re-shared among the others, repeatedly; with no variance left they share
 * equally, with no variance at all every S_k = S), and the real shares x_k
 * become integers as floor(X_k + 1/2) - floor(X_(k-1) + 1/2), X_k the sum of
 * x_1..x_k in slot order.  Var(H_k) = sum over K and V and subspaces g of
 * sum_c P(c) |C_g[c]|^2 - |sum_c P(c) C_g[c]|^2 (clamped at 0), P(c) =
 * H[g][c] / n_res, 0 without residuals: the variance of the residual
 * distribution the histograms describe.  All of it in float64 with sums in
 * slot, subspace, codeword and dim order.  The rows are written, slot k's
 * from row sum_(j<k) S_j of its (layer, kv head). */

/* Copies the pseudo-token count of every slot of the current synthesis:
 * int32 [num_layers][num_kv_heads][capacity] (S_k, or S for every active
 * slot without PROTOKV_FLAG_VAR_ALLOC; 0 for inactive slots); count = that
 * many elements.  Errors: PROTOKV_E_STATE when no synthesis was made since
 * the last fold.  Synchronizes `stream`. */
protokv_status protokv_read_pseudo_counts(protokv_t h, int32_t* dst, size_t count, void* stream);

/* Mass-aware readout (Eq. attn_logit): for every layer l, query token t and
 * query head h, with kv head g = h / (Hq/Hkv):
 *   o = softmax([q K_near^T, q K~^T] / sqrt(D) + [0 ; log n_k]) [V_near ; V~].
 * Needs a synthesis of `stream_id` made after its last fold.
 * q: device [num_layers][tq][num_q_heads][D] in kv_dtype.
 * o: device [num_layers][tq][num_q_heads][D] in kv_dtype.
 * lse: device float32 [num_layers][tq][num_q_heads] (natural-log
 *   log-sum-exp of the biased logits) or NULL.
 * 1 <= tq <= max_query_tokens.
 * With rope_theta > 0 (Sec. 3.3 and the appendix on the RoPE anchor) q is
 * unrotated and query token t is rotated at stream position P + t, P =
 * frames appended * T (the query follows the last frame); near keys sit at
 * their own positions and the pseudo-keys of prototype k at tau_k.  The
 * rotation is the rotate-half form: for i < D/2 the pair (x_i, x_(i+D/2))
 * turns by pos * rope_theta^(-2i/D). */
protokv_status protokv_attend(protokv_t h, int32_t stream_id, const void* q, int32_t tq,
                              void* o, float* lse, void* stream);

/* Bytes of the fixed device array behind protokv_attend_static (64 MiB). */
#define PROTOKV_STATIC_SCRATCH_BYTES (64u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * readout as protokv_attend, same arguments, same result up to the readout
 * tolerance (bitwise equal when the split count is the same), whose
 * kernels keep their scratch -- the per-split partial outputs and (m, l)
 * pairs, and with rope_theta > 0 the rotated query -- in a fixed device
 * array of PROTOKV_STATIC_SCRATCH_BYTES compiled into the library instead of
 * the workspace.  Each device holds its own copy until the process ends
 * (its address is looked up once per device, by protokv_init).  No device
 * memory is allocated or freed and nothing needs clearing: every partial is
 * written before it is read.  The context split count is that of
 * protokv_attend, lowered if needed until units * splits * rows * (D + 2) * 4
 * bytes (rows = tq * Hq / Hkv), plus L * tq * Hq * D * kv bytes with rotary
 * positions, fit the array.
 * Errors: as protokv_attend; PROTOKV_E_UNSUPPORTED when even one split does
 * not fit.  All calls on one device share the array: calls that overlap in
 * time on one device (other streams, other handles, other threads) race and
 * must be serialized by the caller. */
protokv_status protokv_attend_static(protokv_t h, int32_t stream_id, const void* q, int32_t tq,
                                     void* o, float* lse, void* stream);

typedef struct {
  uint64_t frames;          /* frames appended to the stream */
  uint64_t evicted_tokens;  /* tokens folded into the bank, per (layer, kv head) */
  int32_t active_slots;     /* prototypes with n_k > 0, per (layer, kv head) */
  int32_t pending;          /* 1 if an evicted frame awaits protokv_fold */
} protokv_stream_info;

/* Host-side bookkeeping of one stream.  Host only, no device access. */
protokv_status protokv_stream_info_get(protokv_t h, int32_t stream_id, protokv_stream_info* out);

typedef struct {
  uint64_t folds;            /* protokv_fold calls that folded something */
  uint64_t tokens_assigned;  /* (token, layer, kv head) assignments by Eq. 1 */
  uint64_t tokens_seeded;    /* (token, layer, kv head) seeds */
  uint64_t refined;          /* assignments re-scored exactly on a few candidates */
  uint64_t refined_full;     /* assignments re-scored exactly against every slot */
  uint64_t near_ties;        /* assignments whose exact top-2 cost margin < 1e-6 */
  uint64_t touched;          /* (prototype, fold) pairs that absorbed >= 1 token */
  uint64_t aged;             /* maintenance: (prototype, fold) mass decays */
  uint64_t merged;           /* maintenance: prototypes merged into a lower slot */
  uint64_t recycled;         /* maintenance: slots reseeded from the near window */
} protokv_counters;

/* Totals since init.  Synchronizes `stream`. */
protokv_status protokv_get_counters(protokv_t h, protokv_counters* out, void* stream);

/* Copies the last fold's assignment of `stream_id`: int32
 * [num_layers][num_kv_heads][T], slot of each token of the evicted frame
 * (seeded tokens give the slot they seeded).  dst may be host or device
 * memory; count = number of int32 elements.  Synchronizes `stream`. */
protokv_status protokv_read_assignments(protokv_t h, int32_t stream_id, int32_t* dst,
                                        size_t count, void* stream);

/* Copies the PQ codebooks of `stream_id` (as given at init, or learned by
 * the warm-up) to dst (host), float32 [num_layers][num_kv_heads][2][G][C][D/G];
 * count must equal that many floats.  Synchronizes `stream`. */
protokv_status protokv_read_codebooks(protokv_t h, int32_t stream_id, float* dst, size_t count,
                                      void* stream);

/* Bank row layout (bytes) of one prototype slot, PROTOKV_ROW_BYTES each,
 * rows ordered [num_layers][num_kv_heads][capacity]:
 *   0     float32 sum_k[128]      sum of absorbed keys (EMA centres: the centre c)
 *   512   float32 sum_v[128]      (EMA centres: the centre p)
 *   1024  float32 sq_k[128]       sum of squared keys
 *   1536  float32 sq_v[128]
 *   2048  uint32  hist_k[8][16]   H^K[g][c] (entries c >= C are 0)
 *   2560  uint32  hist_v[8][16]
 *   3072  uint32  n               mass n_k (0 = inactive)
 *   3076  uint32  n_res
 *   3080  float32 mu_x, mu_y      running spatial mean
 *   3088  float32 sig_xx, sig_xy, sig_yy
 *   3100  int32   tau             stream position of the last absorbed token
 *   3104  padding to 3200 (the library writes bytes 3104..3135 as zeros) */
#define PROTOKV_ROW_BYTES 3200

/* Copies the bank of `stream_id` (num_layers*num_kv_heads*capacity rows) to
 * dst (host or device); bytes must equal that many PROTOKV_ROW_BYTES.
 * Synchronizes `stream`. */
protokv_status protokv_read_bank(protokv_t h, int32_t stream_id, void* dst, size_t bytes,
                                 void* stream);

/* Copies the current synthesis: keys and values [num_layers][num_kv_heads]
 * [capacity*S][D] in kv_dtype (rows k*S..k*S+S-1 belong to slot k; only the
 * first active_slots*S rows of each (layer, kv head) are defined) and bias
 * float32 [num_layers][num_kv_heads][capacity].  Any pointer may be NULL.
 * Rows the synthesis did not write (bf16 KV) are formed first, on `stream`.
 * Errors: PROTOKV_E_STATE when no synthesis was made since the last fold.
 * Synchronizes `stream`. */
protokv_status protokv_read_pseudo(protokv_t h, void* keys, void* values, float* bias,
                                   void* stream);

/* ---------------------------------------------------------------------------
 * Stream state (checkpoint / resume).  The state of one stream is what Alg.
 * "ProtoKV Streaming Update" carries from one token to the next: the near
 * tier B_near (the ring of the last W frames' exact KV) and the far tier
 * B_far (the prototype bank), together with the stream's PQ codebooks (the
 * appendix "PQ codebook initialization" learns them from the stream) and its
 * position.  A state blob is one contiguous host buffer:
 *
 *   offset 0            protokv_state_header
 *   off_ring_k          kv dtype [units][W+1][T][D]: ring slot f mod (W+1)
 *                       holds frame f of the last W+1 frames appended
 *   off_ring_v          likewise for values
 *   off_bank            [units][capacity] rows of PROTOKV_ROW_BYTES (layout
 *                       above)
 *   off_codebooks       float32 [units][2][G][C][D/G] (as protokv_init takes)
 *   off_reservoir       float32 [units][2][warm_tokens][D]: the warm-up
 *                       reservoir (present when warm_frames > 0, else 0)
 *   off_ring_kr         kv dtype [units][W+1][T][D]: the ring's keys rotated
 *                       at their stream positions (present when
 *                       rope_theta > 0, else 0)
 *
 * units = num_layers * num_kv_heads; every section starts at a multiple of
 * 256 bytes.  The screening copies of the prototype centres are not part of
 * the state: protokv_set_state rebuilds them from the bank rows.
 * --------------------------------------------------------------------------- */
#define PROTOKV_STATE_MAGIC 0x53564B50u /* "PKVS" */
#define PROTOKV_STATE_VERSION 1u

typedef struct {
  uint32_t magic;            /* PROTOKV_STATE_MAGIC */
  uint32_t version;          /* PROTOKV_STATE_VERSION */
  uint32_t units;            /* num_layers * num_kv_heads */
  uint32_t capacity;         /* K */
  uint32_t tokens_per_frame; /* T */
  uint32_t window_frames;    /* W */
  uint32_t kv_bytes;         /* 2 (bf16) or 4 (float32) */
  uint32_t codewords;        /* C */
  uint32_t warm_tokens;      /* reservoir rows per unit (0 when warm_frames = 0) */
  uint32_t rotated;          /* 1 when the rotated-key ring section is present */
  uint64_t frames;           /* frames appended to the stream */
  uint64_t evicted_tokens;   /* tokens folded into each unit's bank */
  int32_t active_slots;      /* slots 0 .. active_slots-1 hold n > 0, the rest n = 0 */
  int32_t folds;             /* folds done (the first warm_frames are the codebook warm-up) */
  int32_t reservoir_rows;    /* warm-up reservoir rows filled per unit */
  int32_t pad;
  uint64_t off_ring_k, off_ring_v, off_bank, off_codebooks, off_reservoir, off_ring_kr;
  uint64_t total_bytes;      /* size of the whole blob */
} protokv_state_header;

/* Size of one stream's state blob for this handle.  Host only. */
protokv_status protokv_state_size(protokv_t h, size_t* bytes);

/* Copies the state of `stream_id` into host_buf (bytes = protokv_state_size).
 * Errors: PROTOKV_E_STATE if the stream has an unfolded eviction.
 * Synchronizes `stream`. */
protokv_status protokv_get_state(protokv_t h, int32_t stream_id, void* host_buf, size_t bytes,
                                 void* stream);

/* Replaces the state of `stream_id` with a blob (bytes = protokv_state_size)
 * made by protokv_get_state on a handle of the same configuration, or built
 * by the caller to the layout above.  Checked on the host before anything
 * is copied (PROTOKV_E_INVALID: wrong magic, version or shape, a count out of
 * range, n > 0 outside the active prefix, a bank inconsistent with the
 * stream position); the stream must have no unfolded eviction
 * (PROTOKV_E_STATE).  Rebuilds the screening copies of every slot from the
 * bank rows and invalidates any synthesis of the stream.  Synchronizes
 * `stream`. */
protokv_status protokv_set_state(protokv_t h, int32_t stream_id, const void* host_buf, size_t bytes,
                                 void* stream);

/* Largest number of evicted tokens per (layer, kv head) a stream may reach:
 * the exact top-S decode multiplies eight factors H + 1 < 2^24 into a
 * 192-bit integer, and a residual count H never exceeds the tokens evicted,
 * so protokv_append_frame rejects (PROTOKV_E_UNSUPPORTED) an append that
 * would make the stream evict more than this.  Host only. */
#define PROTOKV_MAX_EVICTED_TOKENS 16777214ull

/* Kernel ids of protokv_kernel_times. */
enum {
  PROTOKV_K_RING_INSERT = 0,
  PROTOKV_K_SEED = 1,
  PROTOKV_K_SCREEN = 2,          /* assignment and PQ encoding of the evicted tokens */
  PROTOKV_K_AGGREGATE = 3,
  PROTOKV_K_SYNTHESIZE = 4,      /* top-S decoding of the histograms */
  PROTOKV_K_ATTEND = 5,
  PROTOKV_K_ATTEND_MERGE = 6,
  PROTOKV_K_PQ_ENCODE = 7,       /* reserved: PQ encoding runs inside the screen kernel */
  PROTOKV_K_MATERIALIZE = 8,     /* pseudo-token rows and biases (float32 KV) */
  PROTOKV_K_MAINTAIN = 9,        /* prototype maintenance (PROTOKV_FLAG_MAINTENANCE) */
  PROTOKV_K_ROPE_RING = 10,      /* ring insert with the rotated key copy (rope_theta > 0; replaces RING_INSERT) */
  PROTOKV_K_ROPE_Q = 11,         /* rotated query (rope_theta > 0) */
  PROTOKV_K_WARM_COLLECT = 12,   /* warm-up residuals into the reservoir (warm_frames > 0) */
  PROTOKV_K_WARM_KMEANS = 13,    /* codebooks learned from the reservoir (warm_frames > 0) */
  PROTOKV_K_ALLOC = 14,          /* variance-aware pseudo-token counts (PROTOKV_FLAG_VAR_ALLOC) */
  PROTOKV_K_COUNT = 16
};

typedef struct {
  double ms[PROTOKV_K_COUNT];          /* summed device time per kernel */
  uint64_t launches[PROTOKV_K_COUNT];  /* launches timed per kernel */
} protokv_kernel_times;

/* Diagnostics: a nonzero kernel_mask (bit i = protokv_kernel_id i) brackets
 * every launch of the selected kernels on this handle with a pair of HIP
 * events recorded on the launch stream, and clears the totals; 0 stops
 * recording.  The events are created without a system-scope fence, so they
 * add no cache writeback to the timed work.  Host only; creates HIP events on
 * first use. */
protokv_status protokv_profile(protokv_t h, uint32_t kernel_mask);

/* Sums the recorded event pairs into `out` (waits for each end event). */
protokv_status protokv_profile_read(protokv_t h, protokv_kernel_times* out);

/* Message for the last failure on h (or of protokv_init when h is NULL).
 * Valid until the next call on h. */
const char* protokv_last_error(protokv_t h);

#ifdef __cplusplus
}
#endif
#endif /* PROTOKV_H */
