// Internal layout shared by the host library and the HIP kernels of libprotokv.
#pragma once

#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

#include "protokv.h"

namespace pkv {

constexpr int D = 128;     // head dim
constexpr int G = 8;       // PQ subspaces
constexpr int DP = 16;     // dims per subspace
constexpr int CMAX = 16;   // codewords per subspace (storage)
constexpr int SMAX = 16;   // pseudo-tokens per prototype
constexpr int TMAX = 1024; // tokens per frame
constexpr int MAXB = 64;   // streams per launch batch
constexpr int MAX_SPLITS = 16;  // attention context splits (partials storage)
constexpr int MAX_RBLOCKS = 2;  // query-row blocks of 256 per kv head
constexpr int KMAX = 65535;     // prototype slots per unit (slot ids fit 16 bits)
constexpr int PCW = SMAX + 2;   // words per (slot, K/V) decode record: S tuples, no-residual flag, tau (key record) / n (value record)
// The bf16 readout forms pseudo-token rows in LDS from at most PS_SLOTS slots
// per 64-row tile, which holds for S >= PS_MIN_S (64 consecutive rows span
// floor(63 / S) + 2 slots at most); below that the synthesis writes the rows.
constexpr int PS_SLOTS = 14;
constexpr int PS_MIN_S = 5;
constexpr int MT_KMAX = 2048;   // largest capacity the maintenance pass supports (its LDS)
constexpr int AL_KMAX = 4096;   // largest capacity of the variance-aware allocation (its LDS)

// Bank row (one prototype slot), byte offsets; see protokv.h.
constexpr int ROW = PROTOKV_ROW_BYTES;
constexpr int ROW_SUMK = 0, ROW_SUMV = 512, ROW_SQK = 1024, ROW_SQV = 1536;
constexpr int ROW_HK = 2048, ROW_HV = 2560, ROW_META = 3072;

struct RowMeta {
  uint32_t n, n_res;
  float mu_x, mu_y, sxx, sxy, syy;
  int32_t tau;
};
static_assert(sizeof(RowMeta) == 32, "row meta is 32 bytes");

// Screening copy of a slot (derived from its row after every update):
// spatial mean; the quadratic form of (Sigma + rho I)^-1 as a sum of two
// squares, q = (la dx + lb dy)^2 + (lc dy)^2; the frame index of tau; an
// active flag; and eps, a bound on the relative error of the screen's
// float32 spatial term (of d_Mah, or of q itself with squared distances).
// The unit key centre sumK/|sumK| lives beside it as a two-term bf16 split
// (hi + lo).
struct CacheMeta {
  float mu_x, mu_y, la, lb, lc;
  int32_t last_frame;
  uint32_t active;
  float eps;
};
static_assert(sizeof(CacheMeta) == 32, "cache meta is 32 bytes");

// Host-side constants of a handle, passed by value to kernels.
struct Dims {
  int L, Hkv, Hq, T, grid_h, grid_w, W, K, S, C, t_idle, units, streams;
  int kv_fp32;
  uint32_t flags;
  float eta;
  double lambda_sp, lambda_idle, ridge;
  double gamma, eps_k, eps_v;  // maintenance (PROTOKV_FLAG_MAINTENANCE)
  float alpha, beta;           // centre EMA rates (PROTOKV_FLAG_EMA_CENTRES)
  double rope_theta;           // rotary positions in the readout (0 = off)
  int warm_frames, warm_tokens, kmeans_epochs, kmeans_batch;  // codebook warm-up
  int pseudo_max;  // variance-aware allocation: largest S_k
  int max_rows;    // max query rows per kv head (max_query_tokens * Hq / Hkv)
  int max_splits;  // attention context splits (partials storage)
};

// Screening copy of the unit centres in 64-byte pieces: for slot tile
// t = k / 32 and dim chunk c = d / 32, the 32 bf16 components of slot k
// sit together, [t][c][k % 32][d % 32].  The aggregation rewrites a touched
// slot in whole 64-byte sectors (partial sectors cost a read-modify-write
// in memory), and the screen's operand load of one k-step (32 slots x 16
// dims) touches 16 cache lines.  Capacity is padded to K32 = 32 * ceil(K /
// 32) slots per unit.
__host__ __device__ inline int cap32(int K) { return (K + 31) & ~31; }
__host__ __device__ inline size_t chat_offset(int k, int d) {
  return (((size_t)(k >> 5) * 4 + (d >> 5)) * 32 + (k & 31)) * 32 + (d & 31);
}
// Slot k's CacheMeta sits at cmeta[k * CMETA_STRIDE] (the second half of its
// 64 bytes is zero), so its rewrite is a whole sector too.
constexpr int CMETA_STRIDE = 2;

// Device pointers into the caller's workspace.
struct Workspace {
  uint8_t* ring_k;            // [streams][units][W+1][T][D] kv dtype
  uint8_t* ring_v;
  uint8_t* bank;              // [streams][units][K] rows of ROW bytes
  uint16_t* chat_hi;          // [streams][units][K32 / 32][4][32][32] bf16 bits (chat_offset)
  uint16_t* chat_lo;
  CacheMeta* cmeta;           // [streams][units][K][CMETA_STRIDE] (entry 0 used)
  int32_t* assign;            // [streams][units][T]
  float* codebooks;           // [streams][units][2][G][CMAX][DP]
  float* cbhn;                // [streams][units][2][G][CMAX]: |C|^2 / 2 (3e38 for codewords >= C)
  float* cbmax;               // [streams][units][2][G]: an upper bound of max_c |C|
  uint8_t* pk;                // [units][K*S][D] kv dtype (synthesis of one stream)
  uint8_t* pv;
  float* pbias;               // [units][K]
  uint32_t* pcodes;           // [units][K][2][PCW]: decoded top-S code tuples, no-residual flag (word SMAX), tau_k and n (word SMAX + 1 of the key and value record, for the readout's row forming)
  float* part_o;              // [units][max_splits][max_rows][D]
  float* part_ml;             // [units][max_splits][max_rows][2]  (max, sum)
  unsigned long long* counters;  // [16]
  uint32_t* touched;             // [streams][units][K]: folds in which the slot absorbed >= 1 token
  // rotary positions (rope_theta > 0; otherwise null)
  uint8_t* ring_kr;              // [streams][units][W+1][T][D] kv dtype: ring_k rotated at f * T + j
  uint8_t* qrot;                 // [L][max_query_tokens][Hq][D] kv dtype: the query rotated at P + t
  const double* rope_inv;        // [D/2]: theta^(-2i/D)
  // codebook warm-up (warm_frames > 0; otherwise null)
  float* reservoir;              // [streams][units][2][warm_tokens][D]: residuals, eviction order
  // EMA centres (PROTOKV_FLAG_EMA_CENTRES; otherwise null)
  float* ema_res;                // [streams][units][T][2][D]: residuals of the fold's tokens
  // variance-aware allocation (PROTOKV_FLAG_VAR_ALLOC; otherwise null), synthesis of one stream
  int32_t* ps_count;             // [units][K]: S_k (0 for inactive slots)
  int32_t* ps_off;               // [units][K]: first row of slot k, sum of S_j over j < k
  float* prow_bias;              // [units][K*S]: bias of every pseudo-token row
};

enum Counter {
  CNT_REFINED = 0,
  CNT_REFINED_FULL = 1,
  CNT_NEAR_TIES = 2,
  CNT_TOUCHED = 3,
  CNT_AGED = 4,
  CNT_MERGED = 5,
  CNT_RECYCLED = 6,
  CNT_COUNT = 16
};

struct AppendBatch {
  int n;
  int sid[MAXB];
  int slot[MAXB];
  int frame[MAXB];  // index of the appended frame in its stream
};

// One pending eviction per entry.
struct FoldBatch {
  int n;
  int sid[MAXB];
  int slot[MAXB];   // ring slot holding the evicted frame
  int fe[MAXB];     // evicted frame index
  int t[MAXB];      // current frame (the one just appended)
  int nact[MAXB];   // active slots before this fold
  int nseed[MAXB];  // tokens of this frame that seed free slots
  int warm[MAXB];   // warm-up fold: no PQ counts, residuals into the reservoir
  int rfill[MAXB];  // reservoir rows already filled (warm-up folds)
};

// Streams whose warm-up ends with this fold: learn their codebooks from
// `count` reservoir rows.
struct KmeansBatch {
  int n;
  int sid[MAXB];
  int count[MAXB];
};

struct AttendArgs {
  int sid;
  int f_first;      // first near frame
  int n_near;       // near tokens (frames * T)
  int n_far;        // pseudo-tokens (active slots * S)
  int tq;
  int splits;       // context splits per kv head
  int chunk;        // context tokens per split (multiple of 64; rows written, gen 0)
  int near_chunk;   // gen 1: near-window tokens per split (multiple of 64) ...
  int far_chunk;    // ... and pseudo-token rows per split (multiple of 64)
  int gen;          // bf16: pseudo-token rows are formed from centres, codes and codebooks (else read from pk, pv)
  const uint8_t* near_k;  // near-window keys: ring_k, or ring_kr with rotary positions
  const float* rowbias;   // bias per pseudo-token row [units][K*S] (variance-aware allocation), else null
  const void* q;
  void* o;
  float* lse;
};

// 16 bytes per lane from global memory straight into LDS at lds + 16 * lane
// (global_load_lds_dwordx4; M0 holds the wave-uniform LDS byte address, passed
// as an input operand bound to M0 so the compiler sets it and knows it is
// read).  Issued as inline asm so the compiler does not treat later LDS reads
// of other buffers as dependent on it: completion is awaited explicitly with
// wait_vm before the barrier that publishes a tile.
__device__ __forceinline__ void lds_dma16(const void* g, void* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(m0) : "memory");
}
// The value of lane l ^ 32 (the other half of the wave) without an LDS
// round trip: v_permlane32_swap exchanges the upper half of one register
// with the lower half of another, so swapping a register with itself
// gives each half the other's value.  Every lane of the wave takes part.
__device__ __forceinline__ uint32_t xor32_u(uint32_t v) {
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return (__lane_id() & 32) ? r[0] : r[1];
}
__device__ __forceinline__ float xor32(float v) { return __uint_as_float(xor32_u(__float_as_uint(v))); }
__device__ __forceinline__ int xor32(int v) { return (int)xor32_u((uint32_t)v); }

// s_waitcnt vmcnt(n) (expcnt / lgkmcnt not waited for)
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Launchers (fold.hip, query.hip).  Return hipSuccess or the launch error.
hipError_t launch_ring_insert(const Dims& dm, const Workspace& ws, const AppendBatch& ab,
                              const void* k, const void* v, hipStream_t st);
hipError_t launch_seed(const Dims& dm, const Workspace& ws, const FoldBatch& fb, int max_seed,
                       hipStream_t st);
hipError_t launch_screen(const Dims& dm, const Workspace& ws, const FoldBatch& fb,
                         hipStream_t st);
hipError_t launch_aggregate(const Dims& dm, const Workspace& ws, const FoldBatch& fb,
                            hipStream_t st);
hipError_t launch_maintain(const Dims& dm, const Workspace& ws, const FoldBatch& fb, hipStream_t st);
// screening copies of every slot of stream sid rebuilt from its bank rows
hipError_t launch_refresh_all(const Dims& dm, const Workspace& ws, int sid, hipStream_t st);
// centres: also write the biases and the words the readout's row forming
// reads (tau_k, n) into the decode records; wide: some slot may hold more than 65534 residuals (the
// 192-bit path runs too)
hipError_t launch_decode(const Dims& dm, const Workspace& ws, int sid, int n_active, bool centres, bool wide,
                         hipStream_t st);
hipError_t launch_materialize(const Dims& dm, const Workspace& ws, int sid, int n_active, hipStream_t st);
// variance-aware allocation: S_k and row offsets of stream sid's slots from their histograms
hipError_t launch_alloc(const Dims& dm, const Workspace& ws, int sid, int n_active, hipStream_t st);
hipError_t launch_attend(const Dims& dm, const Workspace& ws, const AttendArgs& aa,
                         hipStream_t st);
hipError_t launch_attend_merge(const Dims& dm, const Workspace& ws, const AttendArgs& aa,
                               hipStream_t st);
// rotary positions: the query (tq tokens from q, first position p0) into qrot
// ring insert and the rotated copy in one pass (rope_theta > 0)
hipError_t launch_ring_insert_rope(const Dims& dm, const Workspace& ws, const AppendBatch& ab, const void* k,
                                   const void* v, hipStream_t st);
hipError_t launch_rope_q(const Dims& dm, const Workspace& ws, const void* q, int tq, long long p0,
                         hipStream_t st);
// device address of protokv_attend_static's scratch array on the current
// device (looked up once per device, then cached)
constexpr int MAX_DEVICES = 64;
hipError_t static_scratch_ptr(void** out);
// codebook warm-up (warmup.hip)
hipError_t launch_warm_collect(const Dims& dm, const Workspace& ws, const FoldBatch& fb, hipStream_t st);
hipError_t launch_warm_kmeans(const Dims& dm, const Workspace& ws, const KmeansBatch& kb, hipStream_t st);

}  // namespace pkv
