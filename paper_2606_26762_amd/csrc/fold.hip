// Fold path of libprotokv for gfx950: near-window ring insert, slot seeding,
// assignment screen (bf16 MFMA, rigorous error bound, exact fp64 refine) and
// in-order aggregation of the prototype statistics.
//
// Paper: Section "Online update: eviction, assignment, and prototype
// maintenance" (Eq. 1), Section "Residual Statistics" (PQ residuals) and
// Appendix Algorithm "ProtoKV Streaming Update".  Frame-batched reading: the
// non-seed tokens of an evicted frame are assigned against the bank as it
// stands after seeding, then absorbed per prototype in eviction order.
//
// Every state update below is written as an explicit float32 operation
// sequence (the library is compiled with -ffp-contract=off), so the bank is
// reproducible bit for bit.
#include "pkv_internal.h"

namespace pkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

constexpr float U32 = 5.9604645e-08f;  // 2^-24, unit roundoff of float32

// Bound on |screen cos - exact cos| for the split-bf16 MFMA dot product:
// centre normalisation (<= 9u per component), hi/lo split (2^-18 relative),
// key split for float32 keys (2^-18), fp32 accumulation of <= 384 products
// (<= 384u of sum |K_d c_d| <= |K|), norm of K (8u); ~3.6e-5, taken x4.
constexpr float ECOS = 1.5e-4f;
// A token is a near tie when its exact top-2 cost margin is below this.
constexpr double NEAR_TIE = 1e-6;

__device__ __forceinline__ uint32_t f32_bits(float x) { return __float_as_uint(x); }

// float32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float from_bf16(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Two consecutive KV elements (index e, e+1) as float.
template <int FP32>
__device__ __forceinline__ float2 load2(const uint8_t* base, size_t e) {
  if (FP32) {
    return *reinterpret_cast<const float2*>(base + e * 4);
  } else {
    uint32_t w = *reinterpret_cast<const uint32_t*>(base + e * 2);
    return make_float2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Cell-centre coordinates of token j (float32, same operations as the oracle).
__device__ __forceinline__ void token_xy(int j, int gw, int gh, float& x, float& y) {
  int row = j / gw, col = j - row * gw;
  x = ((float)col + 0.5f) / (float)gw;
  y = ((float)row + 0.5f) / (float)gh;
}

// Rewrites the screening copy of one slot from its (updated) statistics.
// sk = this lane's two components (2*lane, 2*lane+1) of sum_k.
__device__ void refresh_cache(const Dims& dm, float2 sk, const RowMeta& m, size_t slot_index,
                              const Workspace& ws, int lane) {
  float nsq = wave_sum(sk.x * sk.x + sk.y * sk.y);
  float inv = nsq > 0.f ? 1.0f / sqrtf(nsq) : 0.f;
  float cx = sk.x * inv, cy = sk.y * inv;
  uint16_t hx = to_bf16(cx), hy = to_bf16(cy);
  uint16_t lx = to_bf16(cx - from_bf16(hx)), ly = to_bf16(cy - from_bf16(hy));
  reinterpret_cast<uint32_t*>(ws.chat_hi + slot_index * D)[lane] = (uint32_t)hx | ((uint32_t)hy << 16);
  reinterpret_cast<uint32_t*>(ws.chat_lo + slot_index * D)[lane] = (uint32_t)lx | ((uint32_t)ly << 16);
  if (lane == 0) {
    double A = (double)m.sxx + dm.ridge, B = (double)m.sxy, Cc = (double)m.syy + dm.ridge;
    double det = A * Cc - B * B;
    CacheMeta c;
    c.mu_x = m.mu_x;
    c.mu_y = m.mu_y;
    c.qa = (float)(Cc / det);
    c.qb = (float)(-B / det);
    c.qc = (float)(A / det);
    c.last_frame = m.tau / dm.T;
    c.active = m.n > 0 ? 1u : 0u;
    c.pad = 0.f;
    ws.cmeta[slot_index] = c;
  }
}

// ---------------------------------------------------------------------------
// Near ring insert: frame -> ring slot (f mod (W+1)) of each listed stream.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_ring_insert(Dims dm, Workspace ws, AppendBatch ab,
                                                     const uint8_t* k, const uint8_t* v,
                                                     size_t unit_bytes, size_t chunks_per_entry) {
  const size_t total = chunks_per_entry * (size_t)ab.n;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    int e = (int)(i / chunks_per_entry);
    size_t off = (i % chunks_per_entry) * 16;
    size_t unit = off / unit_bytes, within = off % unit_bytes;
    size_t dst = (((size_t)ab.sid[e] * dm.units + unit) * (dm.W + 1) + ab.slot[e]) * unit_bytes + within;
    size_t src = (size_t)e * chunks_per_entry * 16 + off;
    *reinterpret_cast<uint4*>(ws.ring_k + dst) = *reinterpret_cast<const uint4*>(k + src);
    *reinterpret_cast<uint4*>(ws.ring_v + dst) = *reinterpret_cast<const uint4*>(v + src);
  }
}

hipError_t launch_ring_insert(const Dims& dm, const Workspace& ws, const AppendBatch& ab,
                              const void* k, const void* v, hipStream_t st) {
  size_t es = dm.kv_fp32 ? 4 : 2;
  size_t unit_bytes = (size_t)dm.T * D * es;
  size_t chunks = unit_bytes * dm.units / 16;
  size_t total = chunks * ab.n;
  int blocks = (int)std::min<size_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(k_ring_insert, dim3(blocks), dim3(256), 0, st, dm, ws, ab,
                     (const uint8_t*)k, (const uint8_t*)v, unit_bytes, chunks);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Seeding (Initialization): token j < nseed of the evicted frame initialises
// slot nact + j with c <- K, p <- V, n <- 1, mu <- s, Sigma <- I, tau <- pos,
// R <- 0.  One wave per token.
// ---------------------------------------------------------------------------
template <int FP32>
__global__ __launch_bounds__(256) void k_seed(Dims dm, Workspace ws, FoldBatch fb, int blocks_per_unit) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int bu = blockIdx.x / blocks_per_unit;
  const int j = (blockIdx.x % blocks_per_unit) * 4 + wave;
  const int b = bu / dm.units, u = bu % dm.units;
  if (j >= fb.nseed[b]) return;
  const int sid = fb.sid[b];
  const size_t unit = (size_t)sid * dm.units + u;
  const size_t es = FP32 ? 4 : 2;
  const size_t fbase = ((unit * (dm.W + 1) + fb.slot[b]) * dm.T) * (size_t)D;
  const float2 kk = load2<FP32>(ws.ring_k, fbase + (size_t)j * D + 2 * lane);
  const float2 vv = load2<FP32>(ws.ring_v, fbase + (size_t)j * D + 2 * lane);
  (void)es;
  const int slot = fb.nact[b] + j;
  const size_t si = unit * dm.K + slot;
  uint8_t* row = ws.bank + si * ROW;
  reinterpret_cast<float2*>(row + ROW_SUMK)[lane] = kk;
  reinterpret_cast<float2*>(row + ROW_SUMV)[lane] = vv;
  reinterpret_cast<float2*>(row + ROW_SQK)[lane] = make_float2(kk.x * kk.x, kk.y * kk.y);
  reinterpret_cast<float2*>(row + ROW_SQV)[lane] = make_float2(vv.x * vv.x, vv.y * vv.y);
  reinterpret_cast<uint2*>(row + ROW_HK)[lane] = make_uint2(0, 0);
  reinterpret_cast<uint2*>(row + ROW_HV)[lane] = make_uint2(0, 0);
  RowMeta m;
  m.n = 1;
  m.n_res = 0;
  token_xy(j, dm.grid_w, dm.grid_h, m.mu_x, m.mu_y);
  m.sxx = 1.f;
  m.sxy = 0.f;
  m.syy = 1.f;
  m.tau = fb.fe[b] * dm.T + j;
  if (lane == 0) {
    *reinterpret_cast<RowMeta*>(row + ROW_META) = m;
    ws.assign[unit * dm.T + j] = slot;
  }
  refresh_cache(dm, kk, m, si, ws, lane);
}

hipError_t launch_seed(const Dims& dm, const Workspace& ws, const FoldBatch& fb, int max_seed,
                       hipStream_t st) {
  int bpu = (max_seed + 3) / 4;
  dim3 grid(fb.n * dm.units * bpu);
  if (dm.kv_fp32)
    hipLaunchKernelGGL(k_seed<1>, grid, dim3(256), 0, st, dm, ws, fb, bpu);
  else
    hipLaunchKernelGGL(k_seed<0>, grid, dim3(256), 0, st, dm, ws, fb, bpu);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Exact cost of Eq. 1 in float64, same formula and operation order as the
// oracle: cos from sumK, unsquared Mahalanobis with ridge, idle indicator.
// ---------------------------------------------------------------------------
template <int FP32>
__device__ double exact_cost(const Dims& dm, const uint8_t* keyrow, double knorm, double kx, double ky,
                             const uint8_t* row, int t_frame) {
  const float* s = reinterpret_cast<const float*>(row + ROW_SUMK);
  double dot = 0.0, n2 = 0.0;
#pragma unroll 8
  for (int d = 0; d < D; d += 2) {
    float2 kv = load2<FP32>(keyrow, d);
    float2 sv = *reinterpret_cast<const float2*>(s + d);
    dot = dot + (double)kv.x * (double)sv.x;
    dot = dot + (double)kv.y * (double)sv.y;
    n2 = n2 + (double)sv.x * (double)sv.x;
    n2 = n2 + (double)sv.y * (double)sv.y;
  }
  const RowMeta m = *reinterpret_cast<const RowMeta*>(row + ROW_META);
  double denom = knorm * sqrt(n2);
  double cosv = denom > 0.0 ? dot / denom : 0.0;
  double dx = kx - (double)m.mu_x, dy = ky - (double)m.mu_y;
  double A = (double)m.sxx + dm.ridge, B = (double)m.sxy, Cc = (double)m.syy + dm.ridge;
  double det = A * Cc - B * B;
  double q = (Cc * dx * dx - 2.0 * B * dx * dy + A * dy * dy) / det;
  double dm_ = sqrt(q > 0.0 ? q : 0.0);
  double idle = (t_frame - m.tau / dm.T) > dm.t_idle ? 1.0 : 0.0;
  return -cosv + dm.lambda_sp * dm_ + dm.lambda_idle * idle;
}

// Element n of a 4-entry register list (INFINITY / -1 past the end).
__device__ __forceinline__ float pick4(const float* a, int n) {
  return n == 0 ? a[0] : n == 1 ? a[1] : n == 2 ? a[2] : n == 3 ? a[3] : INFINITY;
}
__device__ __forceinline__ int pick4i(const int* a, int n) {
  return n == 0 ? a[0] : n == 1 ? a[1] : n == 2 ? a[2] : n == 3 ? a[3] : -1;
}

// (cost, slot) lexicographic minimum: lower cost, then lower slot.
__device__ __forceinline__ bool better(double c1, int k1, double c2, int k2) {
  return c1 < c2 || (c1 == c2 && k1 < k2);
}

// ---------------------------------------------------------------------------
// Screen + argmin.  Workgroup = 4 waves x 32 tokens; each wave scores its 32
// tokens against every active slot with v_mfma_f32_32x32x16_bf16
// (slots = rows, tokens = columns), slot tiles of 32 staged in LDS.
// Per token it keeps the 4 smallest lower bounds and the smallest upper
// bound of the cost; a token whose bound interval admits a single slot is
// assigned directly, otherwise the candidate slots (or all slots, when more
// than 3 qualify) are re-scored exactly in float64.
// ---------------------------------------------------------------------------
constexpr int SCREEN_TOK = 128;
constexpr int LDS_ROW = 136;  // bf16 per staged row (128 + 8 padding)

template <int FP32>
__global__ __launch_bounds__(256) void k_screen(Dims dm, Workspace ws, FoldBatch fb, int tiles_per_unit) {
  __shared__ __attribute__((aligned(16))) uint16_t s_hi[2][32 * LDS_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t s_lo[2][32 * LDS_ROW];
  __shared__ CacheMeta s_meta[2][32];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tile = blockIdx.x % tiles_per_unit;
  const int bu = blockIdx.x / tiles_per_unit;
  const int b = bu / dm.units, u = bu % dm.units;
  const int N = dm.T;
  const int nseed = fb.nseed[b];
  if (tile * SCREEN_TOK + SCREEN_TOK <= nseed || tile * SCREEN_TOK >= N) return;  // uniform
  const int kact = fb.nact[b] + nseed;
  const int t_frame = fb.t[b];
  const size_t unit = (size_t)fb.sid[b] * dm.units + u;
  const size_t fbase = ((unit * (dm.W + 1) + fb.slot[b]) * N) * (size_t)D;
  const size_t es = FP32 ? 4 : 2;
  const uint8_t* kframe = ws.ring_k + fbase * es;

  const int col = lane & 31, half = lane >> 5;
  const int j = tile * SCREEN_TOK + wave * 32 + col;
  const bool valid = (j >= nseed) && (j < N);
  const int jc = valid ? j : 0;  // any in-bounds row for lanes without a token

  // B operand: K^T (dims x tokens).  Lane holds dims kk*16 + half*8 + 0..7 of token col.
  bf16x8 bk[8];
  bf16x8 bkl[8];
  float nsq = 0.f;
  {
    const uint8_t* kr = kframe + (size_t)jc * D * es;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const int d0 = kk * 16 + half * 8;
      if (FP32) {
        const float4 a0 = *reinterpret_cast<const float4*>(kr + (size_t)d0 * 4);
        const float4 a1 = *reinterpret_cast<const float4*>(kr + (size_t)(d0 + 4) * 4);
        float f[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        u16x8 h, l;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          float x = valid ? f[i] : 0.f;
          nsq += x * x;
          uint16_t hb = to_bf16(x);
          h[i] = hb;
          l[i] = to_bf16(x - from_bf16(hb));
        }
        bk[kk] = __builtin_bit_cast(bf16x8, h);
        bkl[kk] = __builtin_bit_cast(bf16x8, l);
      } else {
        u16x8 h = *reinterpret_cast<const u16x8*>(kr + (size_t)d0 * 2);
        if (!valid) h = (u16x8)0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          float x = from_bf16(h[i]);
          nsq += x * x;
        }
        bk[kk] = __builtin_bit_cast(bf16x8, h);
      }
    }
  }
  nsq += __shfl_xor(nsq, 32, 64);
  const float invn = nsq > 0.f ? 1.0f / sqrtf(nsq) : 0.f;
  float tx, ty;
  token_xy(valid ? j : 0, dm.grid_w, dm.grid_h, tx, ty);

  const float lsp = (float)dm.lambda_sp, lid = (float)dm.lambda_idle;
  float lb[4] = {INFINITY, INFINITY, INFINITY, INFINITY};
  int id[4] = {-1, -1, -1, -1};
  float ubmin = INFINITY;

  const int ntiles = (kact + 31) / 32;
  const uint16_t* ghi = ws.chat_hi + unit * dm.K * D;
  const uint16_t* glo = ws.chat_lo + unit * dm.K * D;
  const CacheMeta* gmeta = ws.cmeta + unit * dm.K;

  auto stage = [&](int t, int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i;         // 0..1023 chunks of 16 B
      const int which = c >> 9;            // 0 = hi, 1 = lo
      const int r = (c & 511) >> 4;        // row 0..31
      const int c16 = c & 15;              // 16-byte column chunk
      const int k = t * 32 + r;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (k < kact) val = *reinterpret_cast<const uint4*>((which ? glo : ghi) + (size_t)k * D + c16 * 8);
      *reinterpret_cast<uint4*>((which ? s_lo[buf] : s_hi[buf]) + r * LDS_ROW + c16 * 8) = val;
    }
    if (tid < 32) {
      const int k = t * 32 + tid;
      CacheMeta cm;
      if (k < kact) cm = gmeta[k];
      else { cm.mu_x = cm.mu_y = cm.qa = cm.qb = cm.qc = cm.pad = 0.f; cm.last_frame = 0; cm.active = 0; }
      s_meta[buf][tid] = cm;
    }
  };

  stage(0, 0);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) stage(t + 1, buf ^ 1);
    f32x16 acc = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const uint16_t* rh = s_hi[buf] + col * LDS_ROW + half * 8;
    const uint16_t* rl = s_lo[buf] + col * LDS_ROW + half * 8;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const bf16x8 ah = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(rh + kk * 16));
      const bf16x8 al = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(rl + kk * 16));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bk[kk], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bk[kk], acc, 0, 0, 0);
      if (FP32) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bkl[kk], acc, 0, 0, 0);
    }
    if (valid) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = (r >> 2) * 8 + half * 4 + (r & 3);
        const int k = t * 32 + m;
        if (k < kact) {
          const CacheMeta cm = s_meta[buf][m];
          const float cosv = acc[r] * invn;
          const float dx = tx - cm.mu_x, dy = ty - cm.mu_y;
          const float t1 = cm.qa * dx * dx;
          const float t2 = (2.0f * cm.qb) * dx * dy;
          const float t3 = cm.qc * dy * dy;
          const float q = t1 + t2 + t3;
          const float qabs = fabsf(t1) + fabsf(t2) + fabsf(t3);
          const float qp = q > 0.f ? q : 0.f;
          const float dd = sqrtf(qp);
          const float eq = 16.0f * U32 * qabs + 1e-30f;
          float ed = qp > eq ? 1.01f * eq * rsqrtf(qp) : sqrtf(eq);
          ed += 2.5e-7f * dd;
          const float idle = (t_frame - cm.last_frame) > dm.t_idle ? 1.f : 0.f;
          const float cost = -cosv + lsp * dd + lid * idle;
          const float e = ECOS + lsp * ed + 4e-7f * (fabsf(cost) + 1.0f);
          const float lo = cost - e, hi = cost + e;
          ubmin = fminf(ubmin, hi);
          if (lo < lb[3]) {
            if (lo < lb[2]) {
              lb[3] = lb[2]; id[3] = id[2];
              if (lo < lb[1]) {
                lb[2] = lb[1]; id[2] = id[1];
                if (lo < lb[0]) { lb[1] = lb[0]; id[1] = id[0]; lb[0] = lo; id[0] = k; }
                else { lb[1] = lo; id[1] = k; }
              } else { lb[2] = lo; id[2] = k; }
            } else { lb[3] = lo; id[3] = k; }
          }
        }
      }
    }
    __syncthreads();
  }

  // Merge with the partner lane holding the other 16 rows of each slot tile.
  {
    float plb[4];
    int pid[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      plb[i] = __shfl_xor(lb[i], 32, 64);
      pid[i] = __shfl_xor(id[i], 32, 64);
    }
    ubmin = fminf(ubmin, __shfl_xor(ubmin, 32, 64));
    float mlb[4];
    int mid[4];
    int na = 0, nb = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float ha = pick4(lb, na), hb = pick4(plb, nb);
      const int ia = pick4i(id, na), ib = pick4i(pid, nb);
      const bool takeA = (ha < hb) || (ha == hb && (unsigned)ia <= (unsigned)ib);
      mlb[i] = takeA ? ha : hb;
      mid[i] = takeA ? ia : ib;
      na += takeA ? 1 : 0;
      nb += takeA ? 0 : 1;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) { lb[i] = mlb[i]; id[i] = mid[i]; }
  }

  const float thr = ubmin + 2e-6f;
  int nc = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) nc += (lb[i] <= thr) ? 1 : 0;
  const bool mine = valid && half == 0;
  if (mine && nc <= 1) ws.assign[unit * N + j] = id[0];
  const bool flag = mine && nc >= 2;

  // Exact refine of flagged tokens, one token at a time per wave.
  unsigned long long fm = __ballot(flag);
  int n_ref = 0, n_full = 0, n_tie = 0;
  while (fm) {
    const int src = __ffsll((long long)fm) - 1;
    fm &= fm - 1;
    const int jj = __shfl(j, src, 64);
    const int ncc = __shfl(nc, src, 64);
    int cand[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) cand[i] = __shfl(id[i], src, 64);
    const uint8_t* kr = kframe + (size_t)jj * D * es;
    float kxf, kyf;
    token_xy(jj, dm.grid_w, dm.grid_h, kxf, kyf);
    double kn2 = 0.0;
    for (int d = 0; d < D; d += 2) {
      float2 kv = load2<FP32>(kr, d);
      kn2 = kn2 + (double)kv.x * (double)kv.x;
      kn2 = kn2 + (double)kv.y * (double)kv.y;
    }
    const double knorm = sqrt(kn2);
    double c1 = INFINITY, c2 = INFINITY;
    int k1 = 0x7fffffff;
    if (ncc <= 3) {
      if (lane < ncc) {
        const int k = cand[lane == 0 ? 0 : lane == 1 ? 1 : 2];
        c1 = exact_cost<FP32>(dm, kr, knorm, kxf, kyf, ws.bank + (unit * dm.K + k) * ROW, t_frame);
        k1 = k;
      }
    } else {
      for (int k = lane; k < kact; k += 64) {
        double c = exact_cost<FP32>(dm, kr, knorm, kxf, kyf, ws.bank + (unit * dm.K + k) * ROW, t_frame);
        if (better(c, k, c1, k1)) { c2 = c1; c1 = c; k1 = k; }
        else if (c < c2) c2 = c;
      }
    }
    // wave reduction of (best, second) with the (cost, slot) order
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      double oc1 = __shfl_xor(c1, o, 64), oc2 = __shfl_xor(c2, o, 64);
      int ok1 = __shfl_xor(k1, o, 64);
      if (better(oc1, ok1, c1, k1)) { c2 = fmin(c1, oc2); c1 = oc1; k1 = ok1; }
      else { c2 = fmin(c2, oc1); }
    }
    if (lane == 0) {
      ws.assign[unit * N + jj] = k1;
      n_ref += 1;
      n_full += ncc > 3 ? 1 : 0;
      n_tie += (c2 - c1) < NEAR_TIE ? 1 : 0;
    }
  }
  if (lane == 0 && n_ref) {
    atomicAdd(&ws.counters[CNT_REFINED], (unsigned long long)(n_ref - n_full));
    if (n_full) atomicAdd(&ws.counters[CNT_REFINED_FULL], (unsigned long long)n_full);
    if (n_tie) atomicAdd(&ws.counters[CNT_NEAR_TIES], (unsigned long long)n_tie);
  }
}

hipError_t launch_screen(const Dims& dm, const Workspace& ws, const FoldBatch& fb, hipStream_t st) {
  int tpu = (dm.T + SCREEN_TOK - 1) / SCREEN_TOK;
  dim3 grid(fb.n * dm.units * tpu);
  if (dm.kv_fp32)
    hipLaunchKernelGGL(k_screen<1>, grid, dim3(256), 0, st, dm, ws, fb, tpu);
  else
    hipLaunchKernelGGL(k_screen<0>, grid, dim3(256), 0, st, dm, ws, fb, tpu);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Aggregation.  Workgroup = 4 waves over a chunk of AGG_KC slots; each wave
// owns whole slots, finds their tokens with ballots over the assignment
// vector (ascending token order) and updates the slot's row in registers:
// lane l holds components 2l, 2l+1 of the sums and histogram bins 2l, 2l+1
// (subspace l/8, codewords 2(l%8), 2(l%8)+1).
// ---------------------------------------------------------------------------
constexpr int AGG_KC = 16;

// Nearest codeword of subspace g = lane/8 for a residual held two components
// per lane.  dist(c) = sum_u (r_u - C[g][c][u])^2 accumulated in float32
// with u ascending; ties go to the lower codeword.
__device__ __forceinline__ int pq_code(float2 r, const float* cb /* [G][CMAX][DP] */, int lane, int C) {
  const int g = lane >> 3;
  float rv[16];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    rv[2 * i] = __shfl(r.x, g * 8 + i, 64);
    rv[2 * i + 1] = __shfl(r.y, g * 8 + i, 64);
  }
  const int c0 = 2 * (lane & 7);
  float best = INFINITY;
  int bc = CMAX;
#pragma unroll
  for (int cc = 0; cc < 2; ++cc) {
    const int c = c0 + cc;
    if (c < C) {
      const float* w = cb + (g * CMAX + c) * DP;
      float acc = 0.f;
#pragma unroll
      for (int uu = 0; uu < DP; ++uu) {
        float dlt = rv[uu] - w[uu];
        float sq = dlt * dlt;
        acc = acc + sq;
      }
      if (acc < best) { best = acc; bc = c; }
    }
  }
#pragma unroll
  for (int o = 1; o <= 4; o <<= 1) {
    float ob = __shfl_xor(best, o, 64);
    int oc = __shfl_xor(bc, o, 64);
    if (ob < best || (ob == best && oc < bc)) { best = ob; bc = oc; }
  }
  return bc;
}

template <int FP32>
__global__ __launch_bounds__(256) void k_aggregate(Dims dm, Workspace ws, FoldBatch fb, int chunks_per_unit) {
  __shared__ float s_cb[2 * G * CMAX * DP];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int chunk = blockIdx.x % chunks_per_unit;
  const int bu = blockIdx.x / chunks_per_unit;
  const int b = bu / dm.units, u = bu % dm.units;
  const int N = dm.T;
  const int nseed = fb.nseed[b];
  const int kact = fb.nact[b] + nseed;
  const int k0 = chunk * AGG_KC;
  if (nseed >= N || k0 >= kact) return;  // uniform
  const size_t unit = (size_t)fb.sid[b] * dm.units + u;
  const bool pq = (dm.flags & PROTOKV_FLAG_PQ) != 0;
  if (pq) {
    const float4* src = reinterpret_cast<const float4*>(ws.codebooks + unit * (2 * G * CMAX * DP));
    for (int i = tid; i < 2 * G * CMAX * DP / 4; i += 256) reinterpret_cast<float4*>(s_cb)[i] = src[i];
  }
  __syncthreads();

  const size_t fbase = ((unit * (dm.W + 1) + fb.slot[b]) * N) * (size_t)D;
  const size_t es = FP32 ? 4 : 2;
  (void)es;
  // assignment of the non-seed tokens, 64 per register
  int areg[TMAX / 64];
#pragma unroll
  for (int c = 0; c < TMAX / 64; ++c) {
    const int jj = c * 64 + lane;
    areg[c] = (jj < N && jj >= nseed) ? ws.assign[unit * N + jj] : -1;
  }
  const float eta = dm.eta, keep = 1.0f - dm.eta;
  int touched = 0;
  for (int i = 0; i < AGG_KC / 4; ++i) {
    const int k = k0 + wave * (AGG_KC / 4) + i;
    if (k >= kact) break;
    unsigned long long masks[TMAX / 64];
    bool any = false;
#pragma unroll
    for (int c = 0; c < TMAX / 64; ++c) {
      masks[c] = (c * 64 < N) ? __ballot(areg[c] == k) : 0ull;
      any |= masks[c] != 0ull;
    }
    if (!any) continue;
    ++touched;
    const size_t si = unit * dm.K + k;
    uint8_t* row = ws.bank + si * ROW;
    float2 sk = reinterpret_cast<const float2*>(row + ROW_SUMK)[lane];
    float2 sv = reinterpret_cast<const float2*>(row + ROW_SUMV)[lane];
    float2 qk = reinterpret_cast<const float2*>(row + ROW_SQK)[lane];
    float2 qv = reinterpret_cast<const float2*>(row + ROW_SQV)[lane];
    uint2 hk = reinterpret_cast<const uint2*>(row + ROW_HK)[lane];
    uint2 hv = reinterpret_cast<const uint2*>(row + ROW_HV)[lane];
    RowMeta m = *reinterpret_cast<const RowMeta*>(row + ROW_META);
    // snapshot centres for the residuals
    const float nf = (float)m.n;
    const float2 cs = make_float2(sk.x / nf, sk.y / nf);
    const float2 ps = make_float2(sv.x / nf, sv.y / nf);
#pragma unroll
    for (int c = 0; c < TMAX / 64; ++c) {
      unsigned long long mk = masks[c];
      while (mk) {
        const int bit = __ffsll((long long)mk) - 1;
        mk &= mk - 1;
        const int jj = c * 64 + bit;
        const float2 kk = load2<FP32>(ws.ring_k, fbase + (size_t)jj * D + 2 * lane);
        const float2 vv = load2<FP32>(ws.ring_v, fbase + (size_t)jj * D + 2 * lane);
        sk.x = sk.x + kk.x; sk.y = sk.y + kk.y;
        sv.x = sv.x + vv.x; sv.y = sv.y + vv.y;
        qk.x = qk.x + kk.x * kk.x; qk.y = qk.y + kk.y * kk.y;
        qv.x = qv.x + vv.x * vv.x; qv.y = qv.y + vv.y * vv.y;
        if (pq) {
          const float2 rk = make_float2(kk.x - cs.x, kk.y - cs.y);
          const float2 rv = make_float2(vv.x - ps.x, vv.y - ps.y);
          const int zk = pq_code(rk, s_cb, lane, dm.C);
          const int zv = pq_code(rv, s_cb + G * CMAX * DP, lane, dm.C);
          const int c0 = 2 * (lane & 7);
          hk.x += (zk == c0) ? 1u : 0u;
          hk.y += (zk == c0 + 1) ? 1u : 0u;
          hv.x += (zv == c0) ? 1u : 0u;
          hv.y += (zv == c0 + 1) ? 1u : 0u;
          m.n_res += 1;
        }
        float sx, sy;
        token_xy(jj, dm.grid_w, dm.grid_h, sx, sy);
        const float mx = keep * m.mu_x + eta * sx;
        const float my = keep * m.mu_y + eta * sy;
        m.mu_x = mx;
        m.mu_y = my;
        const float ddx = sx - mx, ddy = sy - my;
        m.sxx = keep * m.sxx + eta * (ddx * ddx);
        m.sxy = keep * m.sxy + eta * (ddx * ddy);
        m.syy = keep * m.syy + eta * (ddy * ddy);
        m.tau = fb.fe[b] * N + jj;
        m.n += 1;
      }
    }
    reinterpret_cast<float2*>(row + ROW_SUMK)[lane] = sk;
    reinterpret_cast<float2*>(row + ROW_SUMV)[lane] = sv;
    reinterpret_cast<float2*>(row + ROW_SQK)[lane] = qk;
    reinterpret_cast<float2*>(row + ROW_SQV)[lane] = qv;
    reinterpret_cast<uint2*>(row + ROW_HK)[lane] = hk;
    reinterpret_cast<uint2*>(row + ROW_HV)[lane] = hv;
    if (lane == 0) *reinterpret_cast<RowMeta*>(row + ROW_META) = m;
    refresh_cache(dm, sk, m, si, ws, lane);
  }
  if (lane == 0 && touched) atomicAdd(&ws.counters[CNT_TOUCHED], (unsigned long long)touched);
}

hipError_t launch_aggregate(const Dims& dm, const Workspace& ws, const FoldBatch& fb, hipStream_t st) {
  int cpu = (dm.K + AGG_KC - 1) / AGG_KC;
  dim3 grid(fb.n * dm.units * cpu);
  if (dm.kv_fp32)
    hipLaunchKernelGGL(k_aggregate<1>, grid, dim3(256), 0, st, dm, ws, fb, cpu);
  else
    hipLaunchKernelGGL(k_aggregate<0>, grid, dim3(256), 0, st, dm, ws, fb, cpu);
  return hipGetLastError();
}

}  // namespace pkv
