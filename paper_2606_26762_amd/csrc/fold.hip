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
#include <algorithm>

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

// The lane id as a value the compiler cannot see through: per-lane index
// arithmetic derived from it is recomputed where it is used instead of being
// hoisted out of loops and held in registers for the whole kernel.
__device__ __forceinline__ int opaque_lane() {
  int l = (int)(threadIdx.x & 63);
  asm volatile("" : "+v"(l));
  return l;
}

// Sum over the 16 lanes of a lane group (lanes 16m .. 16m+15).
__device__ __forceinline__ float group16_sum(float v) {
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ int group16_sum_i(int v) {
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Cell-centre coordinates of token j (float32, same operations as the oracle).
__device__ __forceinline__ void token_xy(int j, int gw, int gh, float& x, float& y) {
  int row = j / gw, col = j - row * gw;
  x = ((float)col + 0.5f) / (float)gw;
  y = ((float)row + 0.5f) / (float)gh;
}

// Screening meta of a slot from its row meta, in float64.  With
// A = sxx + rho, B = sxy, Cc = syy + rho and det = A Cc - B^2 (> 0), the
// quadratic form of Eq. 1's Mahalanobis distance,
// q = (Cc dx^2 - 2 B dx dy + A dy^2) / det, is (la dx + lb dy)^2 + (lc dy)^2
// with la = sqrt(Cc / det), lb = -(B / Cc) la, lc = 1 / sqrt(Cc).
//
// The screen evaluates it in float32 as dx = tx - mu_x, dy = ty - mu_y,
// u = fma(lb, dy, la dx), q' = fma(u, u, (lc dy)^2), from la, lb, lc rounded
// to float32.  Writing U = la X + lb Y and V = lc Y for the exact
// differences X, Y: |lb Y| <= rho |V| <= rho sqrt(q) with rho = |lb| / lc =
// |B| / sqrt(det), so |la X| <= (1 + rho) sqrt(q).  Every rounding is
// relative (u = 2^-24 each: dx, dy, the three factors, two products, the
// fma), which gives |u' - U| <= (4 + 5 rho) u sqrt(q), |(lc dy)'^2 - V^2| <=
// 7 u V^2 and |q' - q| <= (16 + 10 rho) u q to first order.  The distance
// sqrt(q') (the raw v_sqrt_f32, about 1 ulp) then carries half of that plus
// 2.5e-7; q' < 1e-30 is handled as an absolute 2e-15 in the screen.
__device__ __forceinline__ CacheMeta cache_meta(const Dims& dm, const RowMeta& m) {
  const double A = (double)m.sxx + dm.ridge, B = (double)m.sxy, Cc = (double)m.syy + dm.ridge;
  const double det = A * Cc - B * B;
  // la = Cc / sqrt(Cc det), lb = -B / sqrt(Cc det), lc = 1 / sqrt(Cc): two
  // square roots and two divisions (a few float64 roundings, far below the
  // float32 rounding of the factors)
  const double rd = 1.0 / sqrt(det), rc = 1.0 / sqrt(Cc);
  const double rho = fabs(B) * rd;
  const double u = 0x1p-24;
  const double eq = (16.0 + 10.0 * rho) * u * 1.02;
  CacheMeta c;
  c.mu_x = m.mu_x;
  c.mu_y = m.mu_y;
  c.la = (float)(Cc * rc * rd);
  c.lb = (float)(-B * rc * rd);
  c.lc = (float)rc;
  c.last_frame = m.tau / dm.T;
  c.active = m.n > 0 ? 1u : 0u;
  c.eps = (float)(((dm.flags & PROTOKV_FLAG_MAH_SQUARED) ? eq : 0.5 * eq + 2.5e-7) * 1.001);
  return c;
}

// Rewrites the screening copy of one slot from its (updated) statistics.
// sk = this lane's two components (2*lane, 2*lane+1) of sum_k.
__device__ void refresh_cache(const Dims& dm, float2 sk, const RowMeta& m, size_t unit, int k,
                              const Workspace& ws, int lane) {
  const size_t slot_index = unit * dm.K + k;
  float nsq = wave_sum(sk.x * sk.x + sk.y * sk.y);
  float inv = nsq > 0.f ? 1.0f / sqrtf(nsq) : 0.f;
  float cx = sk.x * inv, cy = sk.y * inv;
  uint16_t hx = to_bf16(cx), hy = to_bf16(cy);
  uint16_t lx = to_bf16(cx - from_bf16(hx)), ly = to_bf16(cy - from_bf16(hy));
  // components 2*lane and 2*lane + 1 are adjacent in the swizzled layout
  const size_t off = unit * (size_t)cap32(dm.K) * D + chat_offset(k, 2 * lane);
  *reinterpret_cast<uint32_t*>(ws.chat_hi + off) = (uint32_t)hx | ((uint32_t)hy << 16);
  *reinterpret_cast<uint32_t*>(ws.chat_lo + off) = (uint32_t)lx | ((uint32_t)ly << 16);
  if (lane == 0) {
    const CacheMeta c = cache_meta(dm, m);
    ws.cmeta[slot_index * CMETA_STRIDE] = c;
  }
  if (lane == 1) ws.cmeta[slot_index * CMETA_STRIDE + 1] = CacheMeta{};
}

// As refresh_cache, for a slot owned by a 16-lane group: s = this lane's
// components [8 il, 8 il + 8) of sum_k.
__device__ void refresh_cache16(const Dims& dm, const float (&s)[8], const RowMeta& m, size_t unit, int k,
                                const Workspace& ws, int il) {
  float part = 0.f;
#pragma unroll
  for (int q = 0; q < 8; ++q) part += s[q] * s[q];
  const float nsq = group16_sum(part);
  const float inv = nsq > 0.f ? 1.0f / sqrtf(nsq) : 0.f;
  u16x8 hi, lo;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const float c = s[q] * inv;
    const uint16_t h = to_bf16(c);
    hi[q] = h;
    lo[q] = to_bf16(c - from_bf16(h));
  }
  // components 8 il .. 8 il + 7 are contiguous in the swizzled layout
  const size_t off = unit * (size_t)cap32(dm.K) * D + chat_offset(k, 8 * il);
  *reinterpret_cast<u16x8*>(ws.chat_hi + off) = hi;
  *reinterpret_cast<u16x8*>(ws.chat_lo + off) = lo;
  if (il == 0) {
    const CacheMeta c = cache_meta(dm, m);
    ws.cmeta[(unit * dm.K + k) * CMETA_STRIDE] = c;
  }
  if (il == 1) ws.cmeta[(unit * dm.K + k) * CMETA_STRIDE + 1] = CacheMeta{};
}

// ---------------------------------------------------------------------------
// Near ring insert: frame -> ring slot (f mod (W+1)) of each listed stream.
// Workgroup = one part of one (batch entry, unit): its frame of K and of V is
// one contiguous block on both sides, split into `parts` equal parts of at
// most 1024 16-byte chunks so that every thread issues all of its (up to
// 4 + 4) loads before its first store.  The frame is read once and the ring
// is read again only W frames later, so both go through nontemporal
// accesses that do not keep the lines in L2.
// ---------------------------------------------------------------------------
constexpr int RING_CHUNKS = 1024;  // 16-byte chunks of K (and of V) per workgroup, at most

__global__ __launch_bounds__(256) void k_ring_insert(Dims dm, Workspace ws, AppendBatch ab,
                                                     const uint8_t* k, const uint8_t* v,
                                                     size_t unit_bytes, int parts) {
  const int part = blockIdx.x % parts, eu = blockIdx.x / parts;
  const int e = eu / dm.units, unit = eu % dm.units;
  const size_t dst = (((size_t)ab.sid[e] * dm.units + unit) * (dm.W + 1) + ab.slot[e]) * unit_bytes;
  const size_t src = ((size_t)e * dm.units + unit) * unit_bytes;
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4* ks = reinterpret_cast<const u32x4*>(k + src);
  const u32x4* vs = reinterpret_cast<const u32x4*>(v + src);
  u32x4* kd = reinterpret_cast<u32x4*>(ws.ring_k + dst);
  u32x4* vd = reinterpret_cast<u32x4*>(ws.ring_v + dst);
  const int n16 = (int)(unit_bytes / 16);
  const int per = (n16 + parts - 1) / parts;  // <= RING_CHUNKS
  const int lo = part * per, hi = min(n16, lo + per);
  // loads unconditional (index clamped into the part, which is never empty)
  // so that all eight are in flight together; stores predicated
  // (named registers, not an array: a private array here gets promoted to LDS)
  const int i0 = lo + (int)threadIdx.x, i1 = i0 + 256, i2 = i0 + 512, i3 = i0 + 768;
  const u32x4 a0 = __builtin_nontemporal_load(ks + min(i0, hi - 1)), a1 = __builtin_nontemporal_load(ks + min(i1, hi - 1));
  const u32x4 a2 = __builtin_nontemporal_load(ks + min(i2, hi - 1)), a3 = __builtin_nontemporal_load(ks + min(i3, hi - 1));
  const u32x4 c0 = __builtin_nontemporal_load(vs + min(i0, hi - 1)), c1 = __builtin_nontemporal_load(vs + min(i1, hi - 1));
  const u32x4 c2 = __builtin_nontemporal_load(vs + min(i2, hi - 1)), c3 = __builtin_nontemporal_load(vs + min(i3, hi - 1));
  if (i0 < hi) { __builtin_nontemporal_store(a0, kd + i0); __builtin_nontemporal_store(c0, vd + i0); }
  if (i1 < hi) { __builtin_nontemporal_store(a1, kd + i1); __builtin_nontemporal_store(c1, vd + i1); }
  if (i2 < hi) { __builtin_nontemporal_store(a2, kd + i2); __builtin_nontemporal_store(c2, vd + i2); }
  if (i3 < hi) { __builtin_nontemporal_store(a3, kd + i3); __builtin_nontemporal_store(c3, vd + i3); }
}

hipError_t launch_ring_insert(const Dims& dm, const Workspace& ws, const AppendBatch& ab,
                              const void* k, const void* v, hipStream_t st) {
  size_t es = dm.kv_fp32 ? 4 : 2;
  size_t unit_bytes = (size_t)dm.T * D * es;   // a multiple of 256
  const int parts = (int)((unit_bytes / 16 + RING_CHUNKS - 1) / RING_CHUNKS);
  hipLaunchKernelGGL(k_ring_insert, dim3(ab.n * dm.units * parts), dim3(256), 0, st, dm, ws, ab,
                     (const uint8_t*)k, (const uint8_t*)v, unit_bytes, parts);
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
  refresh_cache(dm, kk, m, unit, slot, ws, lane);
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
// Screening copies of every slot of one stream's units rebuilt from their bank
// rows (after the stream's state was replaced).  One wave per slot.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_refresh_all(Dims dm, Workspace ws, int sid) {
  const int lane = threadIdx.x & 63;
  const size_t gs = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (gs >= (size_t)dm.units * dm.K) return;
  const int u = (int)(gs / dm.K), k = (int)(gs % dm.K);
  const size_t unit = (size_t)sid * dm.units + u;
  const uint8_t* row = ws.bank + (unit * dm.K + k) * ROW;
  const float2 sk = reinterpret_cast<const float2*>(row + ROW_SUMK)[lane];
  const RowMeta m = *reinterpret_cast<const RowMeta*>(row + ROW_META);
  refresh_cache(dm, sk, m, unit, k, ws, lane);
}

hipError_t launch_refresh_all(const Dims& dm, const Workspace& ws, int sid, hipStream_t st) {
  const size_t slots = (size_t)dm.units * dm.K;
  hipLaunchKernelGGL(k_refresh_all, dim3((unsigned)((slots + 3) / 4)), dim3(256), 0, st, dm, ws, sid);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Exact cost of Eq. 1 in float64, same formula and operation order as the
// oracle: cos from sumK, unsquared Mahalanobis with ridge, idle indicator.
// ---------------------------------------------------------------------------
// Eq. 1 from a float64 dot product K.sumK, |K| and |sumK|^2 (oracle formula and
// operation order for the spatial and idle terms).
__device__ double cost_from_meta(const Dims& dm, double dot, double knorm, double n2, double kx, double ky,
                                 const RowMeta& m, int t_frame) {
  double denom = knorm * sqrt(n2);
  double cosv = denom > 0.0 ? dot / denom : 0.0;
  double dx = kx - (double)m.mu_x, dy = ky - (double)m.mu_y;
  double A = (double)m.sxx + dm.ridge, B = (double)m.sxy, Cc = (double)m.syy + dm.ridge;
  double det = A * Cc - B * B;
  double q = (Cc * dx * dx - 2.0 * B * dx * dy + A * dy * dy) / det;
  double dm_ = (dm.flags & PROTOKV_FLAG_MAH_SQUARED) ? (q > 0.0 ? q : 0.0) : sqrt(q > 0.0 ? q : 0.0);
  double idle = (t_frame - m.tau / dm.T) > dm.t_idle ? 1.0 : 0.0;
  return -cosv + dm.lambda_sp * dm_ + dm.lambda_idle * idle;
}
__device__ double cost_from_dot(const Dims& dm, double dot, double knorm, double n2, double kx, double ky,
                                const uint8_t* row, int t_frame) {
  return cost_from_meta(dm, dot, knorm, n2, kx, ky, *reinterpret_cast<const RowMeta*>(row + ROW_META), t_frame);
}

// Exact cost of Eq. 1 in float64 for one (token, slot), serial over dimensions.
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
  return cost_from_dot(dm, dot, knorm, n2, kx, ky, row, t_frame);
}

// (cost, slot) lexicographic minimum: lower cost, then lower slot.
__device__ __forceinline__ bool better(double c1, int k1, double c2, int k2) {
  return c1 < c2 || (c1 == c2 && k1 < k2);
}

// ---------------------------------------------------------------------------
// PQ residual codes (used by the screen once its tokens are assigned).  The
// code of subspace g is the nearest codeword to the residual r = x - c, with
// c = float32(sum / n) the centre of the token's slot before this fold (IEEE
// division, from the slot's row, which the aggregation rewrites only
// afterwards), under the float32 sequential distance
// dist(c) = sum_u (r_u - C[c][u])^2 (u ascending, one rounding per subtract,
// multiply and add; ties to the lower codeword).  It is found as
// argmax_c (r . C_c - |C_c|^2 / 2) on MFMA with a rigorous error bound; a
// subspace whose best two scores are not separated by the bound is decided
// by the sequential float32 distances themselves.
//
// Lane = (token column col = lane % 32, half = lane / 32 of each subspace's 16
// dims).  For subspaces g0 = 2p, g1 = 2p + 1, v_mfma_f32_32x32x16_bf16
// multiplies A = codebook rows (rows 0-15: C[g0], rows 16-31: C[g1]; block
// diagonal over two k-steps) by B = residual dims (k-step 0: g0, 1: g1), both
// split into hi + lo bf16 (hi*hi + hi*lo + lo*hi), starting from -|C|^2 / 2.
// ---------------------------------------------------------------------------
constexpr int CBW = CMAX * DP;  // floats per (K/V, subspace) codebook block

// v -> hi + lo with hi = bf16(v), lo = bf16(v - hi), both round to nearest
// even; two values per packed conversion, hi read back from its bits
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void split8(const float* v, bf16x8& hi, bf16x8& lo) {
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const bf16x2 h = __builtin_convertvector((f32x2){v[i], v[i + 1]}, bf16x2);
    const uint32_t hb = __builtin_bit_cast(uint32_t, h);
    const bf16x2 l = __builtin_convertvector(
        (f32x2){v[i] - __uint_as_float(hb << 16), v[i + 1] - __uint_as_float(hb & 0xFFFF0000u)}, bf16x2);
    hi[i] = h[0];
    hi[i + 1] = h[1];
    lo[i] = l[0];
    lo[i + 1] = l[1];
  }
}

// Codes of subspaces g0 = 2p, g1 = 2p + 1 for this lane's token from its
// residual halves r[0] (g0) and r[1] (g1) and A-operand codebook row w;
// returns the code of subspace g0 (half 0) or g1 (half 1).  r is formed
// with the centre c' = sum * (1 / n) (a correctly rounded reciprocal, then
// a multiply: |c' - c| <= 3.01 u |c| against c = float32(sum / n)); the
// bound carries that difference through cn (the norm of c' over the
// subspace, from both halves), and the exact fallback forms its residual
// from x, the sums s and n with the IEEE division.  hnp (|C|^2 / 2 of the
// side's codewords, [G][CMAX]) and cmx (max norms, [G]) are the workgroup's
// LDS copies.
__device__ __forceinline__ int pq_pair(const Dims& dm, float pinf, float ninf, const float* cbk, const float* hnp, const float* cmx,
                                       const float (&r)[2][8], const float (&w)[8], const float (&x)[2][8],
                                       const float (&sv)[2][8], float nf, float cn2h0, float cn2h1, int p,
                                       bool valid, int lane) {
  const int col = lane & 31, half = lane >> 5;
  const int g0 = 2 * p, g1 = 2 * p + 1;
  const bf16x8 zero8 = {};
  const bool lowrows = col < 16;
  bf16x8 ah, al, b0h, b0l, b1h, b1l;
  split8(w, ah, al);
  split8(r[0], b0h, b0l);
  split8(r[1], b1h, b1l);
  const bf16x8 a0h = lowrows ? ah : zero8, a0l = lowrows ? al : zero8;
  const bf16x8 a1h = lowrows ? zero8 : ah, a1l = lowrows ? zero8 : al;
  float n0 = 0.f, n1 = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    n0 = fmaf(r[0][i], r[0][i], n0);
    n1 = fmaf(r[1][i], r[1][i], n1);
  }
  // accumulator rows (rr / 4) * 8 + half * 4 + rr % 4: rr < 8 -> codeword of g0, else of g1
  f32x16 acc;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 h = *reinterpret_cast<const float4*>(hnp + (q < 2 ? g0 : g1) * CMAX + (q & 1) * 8 + half * 4);
    acc[4 * q + 0] = -h.x;
    acc[4 * q + 1] = -h.y;
    acc[4 * q + 2] = -h.z;
    acc[4 * q + 3] = -h.w;
  }
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0h, b0h, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0h, b0l, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0l, b0h, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1h, b1h, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1h, b1l, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1l, b1h, acc, 0, 0, 0);

  // best two scores per subspace: 8 codewords here, 8 in the partner lane.
  // Each score carries its codeword in its four low mantissa bits (at most
  // 15 ulp, covered by F below), so max / med3 keep the winner's id too;
  // unused codewords start from -3e38, finite, so no tag makes a NaN.
  float bst1[2], bst2[2];
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    float v1 = -INFINITY, v2 = -INFINITY;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const uint32_t cw = (q >> 2) * 8 + half * 4 + (q & 3);
      const float v = __uint_as_float((__float_as_uint(acc[sub * 8 + q]) & ~15u) | cw);
      v2 = __builtin_amdgcn_fmed3f(v, v1, v2);
      v1 = __builtin_amdgcn_fmed3f(v, v1, pinf);  // max without quieting the tagged value (as low3_push)
    }
    const float o1 = xor32(v1), o2 = xor32(v2);
    bst2[sub] = __builtin_amdgcn_fmed3f(__builtin_amdgcn_fmed3f(v1, o1, ninf), __builtin_amdgcn_fmed3f(v2, o2, pinf), pinf);
    bst1[sub] = __builtin_amdgcn_fmed3f(v1, o1, pinf);
  }
  // lane half 0 settles g0, half 1 settles g1
  const int g = half ? g1 : g0;
  const float v1 = half ? bst1[1] : bst1[0], v2 = half ? bst2[1] : bst2[0];
  float rn2 = half ? n1 : n0;
  rn2 += xor32(half ? n0 : n1);  // the partner's half of subspace g
  // |score - exact| <= F for every codeword: the hi + lo split of both
  // operands leaves <= 3 * 2^-16 |r_u| |C_u| per product (the dropped
  // lo * lo and the two split remainders), summed <= 4.6e-5 |r| |C|; the
  // float32 accumulation over three MFMAs adds <= 51 u (|C|^2 / 2 +
  // |r| |C|), the rounded |C|^2 / 2 <= 9 u |C|^2, the codeword tag <= 15 ulp
  // = 1.8e-6 (|C|^2 / 2 + |r| |C|).  The float32 sequential
  // distances of the codewords differ from the exact ones by <= 19 u D,
  // D <= |r|^2 - 2 score of the runner-up (dlead).  Each term is taken with
  // margin.
  float cn2 = half ? cn2h1 : cn2h0;
  cn2 += xor32(half ? cn2h0 : cn2h1);
  const float rn = sqrtf(rn2) * 1.0001f, cm = cmx[g];
  const float dlead = fmaxf(rn * rn - 2.0f * v2, 0.f) + 1e-30f;
  // ... and <= 3.1 u |c| |C| from the centre c' (taken as 2e-7 |c'| |C|)
  const float F = fmaf(fmaf(5.4e-5f, rn, 2e-7f * sqrtf(cn2) * 1.0001f), cm,
                       fmaf(3.5e-6f, cm * cm, 1.2e-6f * dlead));
  int z = (int)(__float_as_uint(v1) & 15u);
  // not separated: the float32 sequential distances decide, one flagged
  // (token, subspace) at a time for the whole wave (lane % 16 = codeword)
  unsigned long long fm = __ballot(valid && !(v1 - v2 > 2.0f * F));
  while (fm) {
    const int src = __ffsll((long long)fm) - 1;
    fm &= fm - 1;
    const int gs = (src >> 5) ? g1 : g0;   // uniform
    const int tc = src & 31;
    const int cw = lane & 15;
    const float* wc = cbk + gs * CBW + cw * DP;
    // the exact residual x - float32(s / n) of subspace gs, this lane's half
    // (n passes through an empty asm so that the divisions stay in this
    // rarely taken loop rather than being hoisted onto the common path)
    float nfl = nf;
    asm volatile("" : "+v"(nfl));
    float rex[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) rex[i] = (gs == g0) ? x[0][i] - sv[0][i] / nfl : x[1][i] - sv[1][i] / nfl;
    float a = 0.f;
#pragma unroll
    for (int q = 0; q < DP; ++q) {
      const float d = __shfl(rex[q & 7], q < 8 ? tc : tc + 32, 64) - wc[q];
      a = a + d * d;
    }
    if (cw >= dm.C) a = INFINITY;
    int ai = cw;
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) {
      const float oa = __shfl_xor(a, o, 64);
      const int oi = __shfl_xor(ai, o, 64);
      const bool take = oa < a || (oa == a && oi < ai);
      a = take ? oa : a;
      ai = take ? oi : ai;
    }
    if (lane == src) z = ai;
  }
  return z;
}


// ---------------------------------------------------------------------------
// Screen + argmin.  Workgroup = 64 evicted tokens of one unit (two 32-token
// columns per lane, keys staged once in LDS); its SW waves split the slot
// tiles (t = wave, wave + SW, ...) and score them with v_mfma_f32_32x32x16_bf16 (slots = rows, tokens =
// columns; unit centres as a hi + lo bf16 split read in MFMA operand order,
// so each k-step is one contiguous 1 KiB load per wave, and the next tile's
// loads are in flight during this tile's epilogue).  The float32 epilogue
// approximates Eq. 1 per (token, slot) with a rigorous bound on its error
// (relative to the cost, from the largest per-slot bound of the spatial
// term over the unit's slots); each lane keeps, per token, the three
// smallest approximate costs (slots of the first two), folded in from each
// slot tile's three smallest row-tagged costs.  A token whose interval
// admits one slot is assigned directly; two candidates are re-scored exactly
// in float64; three or more send the token to an exact float64 pass over
// every slot.  Workgroups are placed so that the tiles of one unit run on the
// same XCD and share its L2 copy of the centres.
// ---------------------------------------------------------------------------
constexpr int SCREEN_TOK = 64;

struct Top3 {
  float c1, c2, c3;  // three smallest approximate costs
  int i1, i2;        // slots of c1 and c2
  float emax;        // largest relative error bound (eps) of the spatial term over the slots screened
};

__device__ __forceinline__ void top3_push(Top3& a, float c, int k) {
  // slot ids by mask arithmetic (nested selects are otherwise lowered to
  // divergent branches)
  const bool lt1 = c < a.c1, lt2 = c < a.c2;
  const int m1 = -(int)lt1, m2 = -(int)lt2;
  const int s2 = (k & m2) | (a.i2 & ~m2);
  a.i2 = (a.i1 & m1) | (s2 & ~m1);
  a.i1 = (k & m1) | (a.i1 & ~m1);
  a.c3 = __builtin_amdgcn_fmed3f(c, a.c2, a.c3);
  a.c2 = __builtin_amdgcn_fmed3f(c, a.c1, a.c2);
  a.c1 = fminf(a.c1, c);
}

// b's third cost can only be the union's third smallest (it has two smaller
// entries of its own, which the pushes already placed).
__device__ __forceinline__ void top3_merge(Top3& a, const Top3& b) {
  top3_push(a, b.c1, b.i1);
  top3_push(a, b.c2, b.i2);
  a.c3 = fminf(a.c3, b.c3);
  a.emax = fmaxf(a.emax, b.emax);
}

// Approximate cost of one (token, slot) pair, with the slot's row m in the
// slot tile (0..31) in its five low mantissa bits: a change of at most 31
// ulp, which the decision's bound covers, and it lets the three smallest of
// a tile's rows be kept by three min / median operations.  a = (mu_x, mu_y,
// la, lb), c = (lc, lambda_idle * idle), with c.y = 3e38 (finite: the row
// bits must not turn it into a NaN) for rows past the active slots.  The
// spatial term's error is the slot's eps relative to the term (cache_meta);
// SQ: the term is q itself.
constexpr float PAST_ACTIVE = 3e38f;
template <int SQ>
__device__ __forceinline__ float screen_cost(float dot, float invn, float tx, float ty, const float4& a,
                                             const float2& c, int m, float lsp) {
  const float dx = tx - a.x, dy = ty - a.y;
  const float u = fmaf(a.w, dy, a.z * dx);
  const float v = c.x * dy;
  const float q = fmaf(u, u, v * v);  // >= 0: a sum of squares
  float term = q;
  // raw v_sqrt_f32 (about 1 ulp; the bound allows 2.5e-7 relative, and
  // q' < 1e-30 an absolute 2e-15)
  if (!SQ) term = __builtin_amdgcn_sqrtf(q);
  const float cost = fmaf(lsp, term, fmaf(-dot, invn, c.y));
  return __uint_as_float((__float_as_uint(cost) & ~31u) | (uint32_t)m);
}

// Three smallest row-tagged costs of a slot tile.
struct Low3 {
  float c1, c2, c3;
};
// The minimum is taken as a median with -inf, held in a register the
// compiler cannot see into: fminf, or a median with a constant infinity that
// it folds back into one, would first quiet the tagged operand (one more
// instruction per pair).
__device__ __forceinline__ float opaque(float x) {
  asm("" : "+v"(x));
  return x;
}
__device__ __forceinline__ void low3_push(Low3& a, float ninf, float c) {
  a.c3 = __builtin_amdgcn_fmed3f(c, a.c2, a.c3);
  a.c2 = __builtin_amdgcn_fmed3f(c, a.c1, a.c2);
  a.c1 = __builtin_amdgcn_fmed3f(c, a.c1, ninf);
}
// ... folded into the token's running top-3 with their slot ids
__device__ __forceinline__ void low3_fold(Top3& top, const Low3& l, int k0) {
  top3_push(top, l.c1, k0 + (int)(__float_as_uint(l.c1) & 31u));
  top3_push(top, l.c2, k0 + (int)(__float_as_uint(l.c2) & 31u));
  top3_push(top, l.c3, k0 + (int)(__float_as_uint(l.c3) & 31u));
}

// SW waves per workgroup, two waves per SIMD either way: four for small
// grids, one (eight workgroups per CU, whose phases overlap better) for
// launches of many thousand workgroups.
template <int FP32, int SQ, int SW>
__global__ __launch_bounds__(64 * SW, 2) void k_screen(Dims dm, Workspace ws, FoldBatch fb, int tiles_per_unit) {
  static_assert(SW == 1 || SW == 4, "waves per workgroup");
  constexpr int SCREEN_WAVES = SW;
  // token operands of the workgroup in MFMA B order [token half][k-step][lane]
  __shared__ bf16x8 s_bk[2][8][64];
  __shared__ bf16x8 s_bkl[FP32 ? 2 : 1][FP32 ? 8 : 1][64];  // low part of float32 keys
  // The staging and slot-tile arrays (partial squared key norms; per slot
  // row mu_x, mu_y, la, lb and lc, lambda_idle * idle, 3e38 past the
  // active slots) share their LDS with the per-wave top-3 of the decision,
  // which is written only after every wave has left the slot tiles: 18 KiB
  // per one-wave workgroup lets eight of them share a CU.
  constexpr int NSQ_B = SCREEN_WAVES * 2 * 64 * 4, MA_B = SCREEN_WAVES * 32 * 16, MB_B = SCREEN_WAVES * 32 * 8;
  constexpr int TOP_B = SCREEN_WAVES * SCREEN_TOK * (int)sizeof(Top3);
  __shared__ __align__(16) unsigned char s_u[TOP_B > NSQ_B + MA_B + MB_B ? TOP_B : NSQ_B + MA_B + MB_B];
  float(*s_nsq)[2][64] = reinterpret_cast<float(*)[2][64]>(s_u);
  float4(*s_ma)[32] = reinterpret_cast<float4(*)[32]>(s_u + NSQ_B);
  float2(*s_mb)[32] = reinterpret_cast<float2(*)[32]>(s_u + NSQ_B + MA_B);
  Top3(*s_top)[SCREEN_TOK] = reinterpret_cast<Top3(*)[SCREEN_TOK]>(s_u);
  __shared__ int s_asg[SCREEN_TOK];                           // final slot of each token of the tile

  // wave is a compile-time 0 for one-wave workgroups: the loops over a
  // wave's share of k-steps, token halves and jobs then unroll with their
  // loads issued together (a wave index the compiler cannot bound turns
  // each step into a guarded load and a wait of its own)
  const int tid = threadIdx.x, lane = tid & 63, wave = SCREEN_WAVES == 1 ? 0 : tid >> 6;
  // Workgroups are dealt to the 8 XCDs round-robin; logical block lb runs on
  // XCD lb / per, so consecutive logical blocks (the tiles of one unit) share
  // an L2.  Within an XCD the workgroups are dealt round-robin to its four
  // shader engines as well: the tile of logical block lb is rotated by its
  // unit so that an engine is not always handed the same tile of every unit
  // (the ragged last tile costs about half a full one).
  const int nblk = (int)gridDim.x, per = nblk >> 3, bid = (int)blockIdx.x;
  const int lb = bid < per * 8 ? (bid & 7) * per + (bid >> 3) : bid;
  const int bu = lb / tiles_per_unit;
  const int tile = (lb % tiles_per_unit + bu) % tiles_per_unit;
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
  const float lsp = (float)dm.lambda_sp;
  const float lidle = (float)dm.lambda_idle;

  const int ntiles = (kact + 31) / 32;
  const size_t K32 = (size_t)cap32(dm.K);
  const uint16_t* ghi = ws.chat_hi + unit * K32 * D + col * 32 + half * 8;
  const uint16_t* glo = ws.chat_lo + unit * K32 * D + col * 32 + half * 8;
  const CacheMeta* gmeta = ws.cmeta + unit * dm.K * CMETA_STRIDE;

  // operands of slot tile t: k-step kk of lane (col, half) is the 16 bytes
  // of slot 32 t + col at dims 16 kk + 8 half (chat_offset), and that row's
  // meta (mu_x, mu_y, la, lb | lc, last_frame, active, eps), read
  // unconditionally from a row clamped into range (kact >= 1 whenever a tile
  // exists) and converted only where it is used: a load under a divergent
  // branch would be waited for at once, with every operand load before it
  u16x8 ah[8], al[8];
  float4 mr0 = make_float4(0.f, 0.f, 0.f, 0.f);
  float4 mr1 = make_float4(0.f, 0.f, 0.f, 0.f);
  auto load_tile = [&](int t) {
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      ah[kk] = *reinterpret_cast<const u16x8*>(ghi + (size_t)t * 32 * D + (kk >> 1) * 1024 + (kk & 1) * 16);
      al[kk] = *reinterpret_cast<const u16x8*>(glo + (size_t)t * 32 * D + (kk >> 1) * 1024 + (kk & 1) * 16);
    }
    const float* mp = reinterpret_cast<const float*>(gmeta + (size_t)min(t * 32 + col, kact - 1) * CMETA_STRIDE);
    mr0 = *reinterpret_cast<const float4*>(mp);
    mr1 = *reinterpret_cast<const float4*>(mp + 4);
  };
  static_assert(offsetof(CacheMeta, lc) == 16 && offsetof(CacheMeta, last_frame) == 20 &&
                offsetof(CacheMeta, eps) == 28, "meta layout");
  if (wave < ntiles) load_tile(wave);  // in flight while the keys are staged

  // Stage the keys: wave w (< SCREEN_WAVES by the launch) loads k-steps w, w + SCREEN_WAVES, ... of both 32-token halves
  // (tokens tile*64 + h*32 + col, dims 16 kk + 8 half .. + 8) and its partial norms.
  int jt[2];
  bool vt[2];
  const uint8_t* krow[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int j = tile * SCREEN_TOK + h * 32 + col;
    const bool valid = (j >= nseed) && (j < N);
    jt[h] = j;
    vt[h] = valid;
    krow[h] = kframe + (size_t)(valid ? j : 0) * D * es;
  }
  if (FP32) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float nsq = 0.f;
#pragma unroll
      for (int ks = 0; ks < 8 / SCREEN_WAVES; ++ks) {
        const int kk = wave + ks * SCREEN_WAVES;
        const int d0 = kk * 16 + half * 8;
        const float4 a0 = *reinterpret_cast<const float4*>(krow[h] + (size_t)d0 * 4);
        const float4 a1 = *reinterpret_cast<const float4*>(krow[h] + (size_t)(d0 + 4) * 4);
        float f[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        u16x8 hh, ll;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          float x = vt[h] ? f[i] : 0.f;
          nsq += x * x;
          uint16_t hb = to_bf16(x);
          hh[i] = hb;
          ll[i] = to_bf16(x - from_bf16(hb));
        }
        s_bk[h][kk][lane] = __builtin_bit_cast(bf16x8, hh);
        s_bkl[FP32 ? h : 0][FP32 ? kk : 0][lane] = __builtin_bit_cast(bf16x8, ll);
      }
      s_nsq[wave][h][lane] = nsq;
    }
  } else {
    // every key load of the wave in flight before the first is used
    u16x8 kraw[2][8 / SCREEN_WAVES];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ks = 0; ks < 8 / SCREEN_WAVES; ++ks)
        kraw[h][ks] = *reinterpret_cast<const u16x8*>(krow[h] + (size_t)((wave + ks * SCREEN_WAVES) * 16 + half * 8) * 2);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float nsq = 0.f;
#pragma unroll
      for (int ks = 0; ks < 8 / SCREEN_WAVES; ++ks) {
        u16x8 hh = kraw[h][ks];
        if (!vt[h]) hh = (u16x8)0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          float x = from_bf16(hh[i]);
          nsq += x * x;
        }
        s_bk[h][wave + ks * SCREEN_WAVES][lane] = __builtin_bit_cast(bf16x8, hh);
      }
      s_nsq[wave][h][lane] = nsq;
    }
  }
  __syncthreads();
  float invn[2], tx[2], ty[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    float nsq = 0.f;
#pragma unroll
    for (int w = 0; w < SCREEN_WAVES; ++w) nsq += s_nsq[w][h][col] + s_nsq[w][h][col + 32];
    invn[h] = nsq > 0.f ? 1.0f / sqrtf(nsq) : 0.f;
    token_xy(vt[h] ? jt[h] : 0, dm.grid_w, dm.grid_h, tx[h], ty[h]);
  }

  Top3 top[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    top[h].c1 = top[h].c2 = top[h].c3 = INFINITY;
    top[h].i1 = top[h].i2 = -1;
    top[h].emax = 0.f;
  }

  // a second token half with no token to screen (the ragged end of a frame:
  // tokens [tile * 64 + 32, tile * 64 + 64) all below nseed or past N)
  // skips its MFMAs and epilogue rows
  const bool live1 = max(tile * SCREEN_TOK + 32, nseed) < min(tile * SCREEN_TOK + SCREEN_TOK, N);  // uniform
  float emx = 0.f;  // largest eps of this lane's rows
  const float ninf = opaque(-INFINITY);
  for (int t = wave; t < ntiles; t += SCREEN_WAVES) {
    if (half == 0) {
      // rows past the active slots: +inf idle term, never selected
      const bool mv = t * 32 + col < kact;
      const bool idle = (t_frame - __float_as_int(mr1.y)) > dm.t_idle;
      s_ma[wave][col] = mv ? mr0 : make_float4(0.f, 0.f, 0.f, 0.f);
      s_mb[wave][col] = mv ? make_float2(mr1.x, idle ? lidle : 0.f) : make_float2(0.f, PAST_ACTIVE);
      emx = fmaxf(emx, mv ? mr1.w : 0.f);
    }
    f32x16 acc0 = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    f32x16 acc1 = acc0;
    // the two halves' products (a half's MFMA chain depends only on itself)
    auto products = [&](int h, f32x16& acc) {
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const bf16x8 xh = __builtin_bit_cast(bf16x8, ah[kk]), xl = __builtin_bit_cast(bf16x8, al[kk]);
        const bf16x8 bk = s_bk[h][kk][lane];
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xh, bk, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xl, bk, acc, 0, 0, 0);
        if (FP32) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xh, s_bkl[FP32 ? h : 0][FP32 ? kk : 0][lane], acc, 0, 0, 0);
      }
    };
    if (live1) {
      // both chains interleaved
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const bf16x8 xh = __builtin_bit_cast(bf16x8, ah[kk]), xl = __builtin_bit_cast(bf16x8, al[kk]);
        const bf16x8 b0 = s_bk[0][kk][lane], b1 = s_bk[1][kk][lane];
        acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xh, b0, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xh, b1, acc1, 0, 0, 0);
        acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xl, b0, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xl, b1, acc1, 0, 0, 0);
        if (FP32) {
          const bf16x8 c0 = s_bkl[FP32 ? 0 : 0][FP32 ? kk : 0][lane];
          const bf16x8 c1 = s_bkl[FP32 ? 1 : 0][FP32 ? kk : 0][lane];
          acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xh, c0, acc0, 0, 0, 0);
          acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xh, c1, acc1, 0, 0, 0);
        }
      }
    } else {
      products(0, acc0);
    }
    if (t + SCREEN_WAVES < ntiles) load_tile(t + SCREEN_WAVES);  // in flight during the epilogue
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    Low3 l0 = {INFINITY, INFINITY, INFINITY}, l1 = l0;
    if (live1) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = (r >> 2) * 8 + half * 4 + (r & 3);
        const float4 a = s_ma[wave][m];
        const float2 c = s_mb[wave][m];
        low3_push(l0, ninf, screen_cost<SQ>(acc0[r], invn[0], tx[0], ty[0], a, c, m, lsp));
        low3_push(l1, ninf, screen_cost<SQ>(acc1[r], invn[1], tx[1], ty[1], a, c, m, lsp));
        if ((r & 3) == 3) __builtin_amdgcn_sched_barrier(0);
      }
      low3_fold(top[0], l0, t * 32);
      low3_fold(top[1], l1, t * 32);
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = (r >> 2) * 8 + half * 4 + (r & 3);
        const float4 a = s_ma[wave][m];
        const float2 c = s_mb[wave][m];
        low3_push(l0, ninf, screen_cost<SQ>(acc0[r], invn[0], tx[0], ty[0], a, c, m, lsp));
        if ((r & 7) == 7) __builtin_amdgcn_sched_barrier(0);
      }
      low3_fold(top[0], l0, t * 32);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // every token's spatial error bound: the largest eps over the wave's rows
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) emx = fmaxf(emx, __shfl_xor(emx, o, 64));
  top[0].emax = top[1].emax = emx;

  // The PQ tail's per-unit constants (both sides' codeword half norms and
  // max norms), fetched now so that the decision covers their latency and
  // staged in LDS once the decision is done.
  const bool pq_on = (dm.flags & (PROTOKV_FLAG_PQ | PROTOKV_FLAG_EMA_CENTRES)) == PROTOKV_FLAG_PQ && !fb.warm[b];
  static_assert(2 * G * CMAX == 64 * 4 && 2 * G <= 4 * 4, "one float4 of half norms per lane, max norms in 4");
  float4 pq_hn = make_float4(0.f, 0.f, 0.f, 0.f), pq_cm = pq_hn;
  if (pq_on && wave == 0) {  // uniform
    pq_hn = reinterpret_cast<const float4*>(ws.cbhn + unit * 2 * G * CMAX)[lane];
    pq_cm = reinterpret_cast<const float4*>(ws.cbmax + unit * 2 * G)[lane & 3];
  }

  // merge with the partner lane (other 16 rows of each slot tile), then
  // across waves (s_top reuses the slot-tile arrays: every wave leaves the
  // slot tiles first)
  if (SCREEN_WAVES > 1) __syncthreads();
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    Top3 o;
    o.c1 = xor32(top[h].c1);
    o.c2 = xor32(top[h].c2);
    o.c3 = xor32(top[h].c3);
    o.i1 = xor32(top[h].i1);
    o.i2 = xor32(top[h].i2);
    o.emax = xor32(top[h].emax);
    top3_merge(top[h], o);
    if (half == 0) s_top[wave][h * 32 + col] = top[h];
  }
  __syncthreads();
  // waves 0 and 1 decide for token columns 0..31 and 32..63 (one wave: both)
  constexpr int HSTEP = SCREEN_WAVES >= 2 ? 2 : 1;
  for (int hsel = wave; hsel < 2; hsel += HSTEP) {  // uniform
  Top3 tp = s_top[0][hsel * 32 + col];
#pragma unroll
  for (int w = 1; w < SCREEN_WAVES; ++w) top3_merge(tp, s_top[w][hsel * 32 + col]);
  const int j = hsel ? jt[1] : jt[0];
  const bool valid = hsel ? vt[1] : vt[0];

  // |cost - cost_exact| <= E(cost) for every slot, with
  // E(c) = E0 + ee max(c + 1.001, 0): ECOS for the dot product, 4e-7
  // (2 + lambda_idle) for rounding the rest of the assembly, lsp 1e-14 for
  // q' < 1e-30, and for the spatial term lsp eps_k s_k <= ee (cost + 1.001)
  // (s_k the term: cost >= -1 + lsp s_k, since cos <= 1 and the idle term
  // is >= 0), ee covering eps_k and the rounding of lsp s_k; the row tag
  // (<= 31 ulp = 3.7e-6 |c|) adds 4.2e-6 to E0 and 3.8e-6 to ee.  c - E(c)
  // is increasing, so slot k can be the exact argmin only if
  // c_k - E(c_k) <= c1 + E(c1), and if the third smallest fails that
  // test, so does every slot after it.  Costs of 1e38 and more are rows
  // past the active slots.
  const float E0 = ECOS + 4e-7f * (2.0f + lidle) + 1e-14f * lsp + 4.2e-6f;
  const float ee = 1.02f * tp.emax + 2.0f * U32 + 3.8e-6f;
  const float thr = tp.c1 + E0 + ee * fmaxf(tp.c1 + 1.001f, 0.f) + 2e-6f;
  const bool cand2 = tp.c2 < 1e38f && tp.c2 - (E0 + ee * fmaxf(tp.c2 + 1.001f, 0.f)) <= thr;
  const bool cand3 = tp.c3 < 1e38f && tp.c3 - (E0 + ee * fmaxf(tp.c3 + 1.001f, 0.f)) <= thr;
  const int nc = 1 + cand2 + cand3;
  const bool mine = valid && half == 0;
  if (mine && nc <= 1) {
    ws.assign[unit * N + j] = tp.i1;
    s_asg[hsel * 32 + col] = tp.i1;
  }
  const bool flag = mine && nc >= 2;

  // Exact refine of flagged tokens, one token at a time.
  unsigned long long fm = __ballot(flag);
  int n_ref = 0, n_full = 0, n_tie = 0;
  while (fm) {
    const int src = __ffsll((long long)fm) - 1;
    fm &= fm - 1;
    const int jj = __shfl(j, src, 64);
    const int ncc = __shfl(nc, src, 64);
    const int cand0 = __shfl(tp.i1, src, 64), cand1 = __shfl(tp.i2, src, 64);
    const uint8_t* kr = kframe + (size_t)jj * D * es;
    float kxf, kyf;
    token_xy(jj, dm.grid_w, dm.grid_h, kxf, kyf);
    double c1 = INFINITY, c2 = INFINITY;
    int k1 = 0x7fffffff;
    if (ncc == 2) {
      // lanes over dimensions: float64 dot products and norms of the two
      // candidates; the key (bf16: from its LDS copy), both sums and both
      // metas in one round trip
      const uint8_t* r0 = ws.bank + (unit * dm.K + cand0) * ROW;
      const uint8_t* r1 = ws.bank + (unit * dm.K + cand1) * ROW;
      const float2 s0 = reinterpret_cast<const float2*>(r0 + ROW_SUMK)[lane];
      const float2 s1 = reinterpret_cast<const float2*>(r1 + ROW_SUMK)[lane];
      const RowMeta m0 = *reinterpret_cast<const RowMeta*>(r0 + ROW_META);
      const RowMeta m1 = *reinterpret_cast<const RowMeta*>(r1 + ROW_META);
      float2 kv;
      if (FP32) {
        kv = load2<FP32>(kr, 2 * lane);
      } else {
        // dims 2l, 2l+1 sit in k-step l / 8, lane half (l / 4) % 2, pair (l % 4)
        const int tl = jj - tile * SCREEN_TOK;
        const uint32_t w = reinterpret_cast<const uint32_t*>(&s_bk[tl >> 5][lane >> 3][((lane >> 2) & 1) * 32 + (tl & 31)])[lane & 3];
        kv = make_float2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
      }
      double kn2 = (double)kv.x * (double)kv.x + (double)kv.y * (double)kv.y;
      double d0 = (double)kv.x * (double)s0.x + (double)kv.y * (double)s0.y;
      double d1 = (double)kv.x * (double)s1.x + (double)kv.y * (double)s1.y;
      double n0 = (double)s0.x * (double)s0.x + (double)s0.y * (double)s0.y;
      double n1 = (double)s1.x * (double)s1.x + (double)s1.y * (double)s1.y;
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) {
        kn2 += __shfl_xor(kn2, o, 64);
        d0 += __shfl_xor(d0, o, 64);
        d1 += __shfl_xor(d1, o, 64);
        n0 += __shfl_xor(n0, o, 64);
        n1 += __shfl_xor(n1, o, 64);
      }
      const double knorm = sqrt(kn2);
      const double e0 = cost_from_meta(dm, d0, knorm, n0, kxf, kyf, m0, t_frame);
      const double e1 = cost_from_meta(dm, d1, knorm, n1, kxf, kyf, m1, t_frame);
      if (better(e0, cand0, e1, cand1)) { c1 = e0; k1 = cand0; c2 = e1; }
      else { c1 = e1; k1 = cand1; c2 = e0; }
    } else {
      double kn2 = 0.0;
      for (int d = 0; d < D; d += 2) {
        float2 kv = load2<FP32>(kr, d);
        kn2 = kn2 + (double)kv.x * (double)kv.x;
        kn2 = kn2 + (double)kv.y * (double)kv.y;
      }
      const double knorm = sqrt(kn2);
      for (int k = lane; k < kact; k += 64) {
        double c = exact_cost<FP32>(dm, kr, knorm, kxf, kyf, ws.bank + (unit * dm.K + k) * ROW, t_frame);
        if (better(c, k, c1, k1)) { c2 = c1; c1 = c; k1 = k; }
        else if (c < c2) c2 = c;
      }
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) {
        double oc1 = __shfl_xor(c1, o, 64), oc2 = __shfl_xor(c2, o, 64);
        int ok1 = __shfl_xor(k1, o, 64);
        if (better(oc1, ok1, c1, k1)) { c2 = fmin(c1, oc2); c1 = oc1; k1 = ok1; }
        else { c2 = fmin(c2, oc1); }
      }
    }
    if (lane == 0) {
      ws.assign[unit * N + jj] = k1;
      s_asg[jj - tile * SCREEN_TOK] = k1;
      n_ref += 1;
      n_full += ncc > 2 ? 1 : 0;
      n_tie += (c2 - c1) < NEAR_TIE ? 1 : 0;
    }
  }
  if (lane == 0 && n_ref) {
    atomicAdd(&ws.counters[CNT_REFINED], (unsigned long long)(n_ref - n_full));
    if (n_full) atomicAdd(&ws.counters[CNT_REFINED_FULL], (unsigned long long)n_full);
    if (n_tie) atomicAdd(&ws.counters[CNT_NEAR_TIES], (unsigned long long)n_tie);
  }
  }  // token halves

  // PQ codes of the tile's assigned tokens: job j = 0..3 (taken by waves
  // j, j + SW, ...) encodes the 32-token block j / 2 of K (j even) or V; each code bumps its bin of the slot's
  // histogram (integer counts: the order of the increments does not matter).
  // With EMA centres the residuals follow each token's own centre update and
  // the aggregation codes them; codebook warm-up folds count no codes.
  if (pq_on) {
    __syncthreads();
    // the decision no longer reads s_top: it holds the unit's half norms
    // [kv][g][CMAX], then its max norms [kv][g]
    static_assert(TOP_B >= (2 * G * CMAX + 2 * G) * (int)sizeof(float), "PQ constants fit s_top");
    float* s_pqc = reinterpret_cast<float*>(s_u);
    if (wave == 0) {
      reinterpret_cast<float4*>(s_pqc)[lane] = pq_hn;
      if (lane < 4) reinterpret_cast<float4*>(s_pqc + 2 * G * CMAX)[lane] = pq_cm;
    }
    __syncthreads();
    for (int job = wave; job < 4; job += SCREEN_WAVES) {  // uniform
    const int blk = job >> 1, kv = job & 1;
    const int jq = tile * SCREEN_TOK + blk * 32 + col;
    const bool qv = jq >= nseed && jq < N;
    if (__ballot(qv)) {  // uniform per wave
      const int slot = qv ? s_asg[blk * 32 + col] : 0;
      const uint8_t* srow = ws.bank + (unit * dm.K + slot) * ROW;
      const float* sums = reinterpret_cast<const float*>(srow + (kv ? ROW_SUMV : ROW_SUMK));
      const size_t ub = unit * 2 + kv;
      const float* cbk = ws.codebooks + ub * G * CBW;
      // every load of the four subspace pairs up front: the token's dims
      // (half of each subspace), the slot's sums of the same dims, n and the
      // A-operand codebook rows
      uint4 xr[G][FP32 ? 2 : 1];
      if (kv == 0 && !FP32) {
#pragma unroll
        for (int g = 0; g < G; ++g) xr[g][0] = __builtin_bit_cast(uint4, s_bk[blk][g][half * 32 + col]);
      } else {
        const uint8_t* xrow = (kv ? ws.ring_v : ws.ring_k) + (fbase + (size_t)(qv ? jq : 0) * D) * es;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const uint4* px = reinterpret_cast<const uint4*>(xrow + (size_t)(g * DP + half * 8) * es);
#pragma unroll
          for (int e = 0; e < (FP32 ? 2 : 1); ++e) xr[g][e] = px[e];
        }
      }
      float4 sr[G][2], wr[G / 2][2];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        sr[g][0] = *reinterpret_cast<const float4*>(sums + g * DP + half * 8);
        sr[g][1] = *reinterpret_cast<const float4*>(sums + g * DP + half * 8 + 4);
      }
#pragma unroll
      for (int p = 0; p < G / 2; ++p) {
        const float* wa = cbk + (2 * p + (col < 16 ? 0 : 1)) * CBW + (col & 15) * DP + half * 8;
        wr[p][0] = *reinterpret_cast<const float4*>(wa);
        wr[p][1] = *reinterpret_cast<const float4*>(wa + 4);
      }
      const float nf = (float)*reinterpret_cast<const uint32_t*>(srow + ROW_META);
      const float inv = 1.0f / nf;
      uint32_t* hist = reinterpret_cast<uint32_t*>(ws.bank + (unit * dm.K + slot) * ROW + (kv ? ROW_HV : ROW_HK));
      const float pinf = opaque(INFINITY);
#pragma unroll
      for (int p = 0; p < G / 2; ++p) {
        float r[2][8], w[8], xs[2][8], ss[2][8], cn2[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int g = 2 * p + q;
          float x[8];
          if (FP32) {
            const uint4 a = xr[g][0], c = xr[g][FP32 ? 1 : 0];
            const uint32_t xw[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
#pragma unroll
            for (int i = 0; i < 8; ++i) x[i] = __uint_as_float(xw[i]);
          } else {
            const uint4 a = xr[g][0];
            const uint32_t xw[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              x[2 * i] = __uint_as_float(xw[i] << 16);
              x[2 * i + 1] = __uint_as_float(xw[i] & 0xFFFF0000u);
            }
          }
          const float sv[8] = {sr[g][0].x, sr[g][0].y, sr[g][0].z, sr[g][0].w,
                               sr[g][1].x, sr[g][1].y, sr[g][1].z, sr[g][1].w};
          float c2 = 0.f;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const float c = sv[i] * inv;
            c2 = fmaf(c, c, c2);
            r[q][i] = x[i] - c;  // garbage for lanes past the frame, which code nothing
            xs[q][i] = x[i];
            ss[q][i] = sv[i];
          }
          cn2[q] = c2;
        }
        w[0] = wr[p][0].x; w[1] = wr[p][0].y; w[2] = wr[p][0].z; w[3] = wr[p][0].w;
        w[4] = wr[p][1].x; w[5] = wr[p][1].y; w[6] = wr[p][1].z; w[7] = wr[p][1].w;
        const int z = pq_pair(dm, pinf, ninf, cbk, s_pqc + kv * G * CMAX, s_pqc + 2 * G * CMAX + kv * G, r, w, xs, ss, nf, cn2[0], cn2[1],
                              p, qv, lane);
        if (qv) atomicAdd(hist + (2 * p + half) * CMAX + z, 1u);
      }
    }
    }
  }
}

hipError_t launch_screen(const Dims& dm, const Workspace& ws, const FoldBatch& fb, hipStream_t st) {
  int tpu = (dm.T + SCREEN_TOK - 1) / SCREEN_TOK;
  const int nwg = fb.n * dm.units * tpu;
  dim3 grid(nwg);
  using KFn = void (*)(Dims, Workspace, FoldBatch, int);
  const bool sq = (dm.flags & PROTOKV_FLAG_MAH_SQUARED) != 0;
  if (nwg >= 8192) {
    const KFn fn = dm.kv_fp32 ? (sq ? k_screen<1, 1, 1> : k_screen<1, 0, 1>) : (sq ? k_screen<0, 1, 1> : k_screen<0, 0, 1>);
    hipLaunchKernelGGL(fn, grid, dim3(64), 0, st, dm, ws, fb, tpu);
  } else {
    const KFn fn = dm.kv_fp32 ? (sq ? k_screen<1, 1, 4> : k_screen<1, 0, 4>) : (sq ? k_screen<0, 1, 4> : k_screen<0, 0, 4>);
    hipLaunchKernelGGL(fn, grid, dim3(256), 0, st, dm, ws, fb, tpu);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Aggregation.  Workgroup = 32 consecutive slots of one unit, two per 16-lane
// group (absorbed one after the other); lane il of a group holds dims
// [8 il, 8 il + 8) of the slot's four sums.  The unit's assignment vector
// is staged in LDS; wave w sweeps it with ballots for its eight slots, once
// to count their tokens and once to list them in eviction order.  A workgroup whose slots drew no token
// exits there.  Each group then loads its slot's row, absorbs the slot's
// tokens in order, TOK_BATCH at a time with all of a batch's loads in flight
// (mass, sums, sums of squares, residual count, spatial EMA, recency; the
// screen already counted the PQ codes into the histograms), writes the row
// back and refreshes the slot's screening copy.  With EMA centres (EMA = 1)
// the sums are the centres, updated per token at rates alpha, beta; each
// token's residuals against its updated centres go to the workspace, and
// once every slot of the workgroup is done, all its threads code every
// (token, K/V, subspace) in parallel and each group adds its slots' codes
// to their histograms.
// ---------------------------------------------------------------------------
// slots per workgroup: NP per 16-lane group (k0 + g + 16 p, p < NP), 16 NP in all
constexpr int AGG_NP = 2;
constexpr int AGG_TOK_BYTES = 32768;  // LDS for the workgroup's tokens (64 bf16 or 32 float32 tokens)
constexpr int TOK_BATCH = 2;
constexpr uint16_t NO_SLOT = 0xFFFF;

// Eight consecutive KV elements (index e, a multiple of 8) as raw words
// (bf16 pairs or float32 bits), and element q of them as float.
template <int FP32>
struct Raw8 {
  uint4 w[FP32 ? 2 : 1];
};
template <int FP32>
// (nontemporal: an evicted token is absorbed once, so its lines need not stay in L2)
__device__ __forceinline__ void load8(const uint8_t* base, size_t e, Raw8<FP32>& x) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4* p = reinterpret_cast<const u32x4*>(base + e * (FP32 ? 4 : 2));
#pragma unroll
  for (int q = 0; q < (FP32 ? 2 : 1); ++q) {
    const u32x4 t = __builtin_nontemporal_load(p + q);
    x.w[q] = make_uint4(t.x, t.y, t.z, t.w);
  }
}
template <int FP32>
__device__ __forceinline__ float raw_at(const Raw8<FP32>& x, int q) {
  const uint4& v = x.w[FP32 ? q >> 2 : 0];
  const int e = FP32 ? (q & 3) : (q >> 1);
  const uint32_t word = e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w;
  if (FP32) return __uint_as_float(word);
  return __uint_as_float((q & 1) ? (word & 0xFFFF0000u) : (word << 16));
}

__device__ __forceinline__ void ld8f(const uint8_t* p, float (&x)[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
// (nontemporal: a rewritten bank row is read again only when a later fold
// touches the slot, long after it has left L2)
__device__ __forceinline__ void st8f(uint8_t* p, const float (&x)[8]) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store((f32x4){x[0], x[1], x[2], x[3]}, reinterpret_cast<f32x4*>(p));
  __builtin_nontemporal_store((f32x4){x[4], x[5], x[6], x[7]}, reinterpret_cast<f32x4*>(p) + 1);
}

template <int FP32, int EMA, int NP>
__global__ __launch_bounds__(256, EMA ? 2 : (NP > 2 ? 3 : 4)) void k_aggregate(Dims dm, Workspace ws, FoldBatch fb,
                                                                            int wg_per_unit) {
  constexpr int AGG_SLOTS = 16 * NP;
  constexpr int NGW = 4 * NP;              // (group, pass) pairs of one wave
  __shared__ uint16_t s_asg[TMAX];         // slot of each token (NO_SLOT: seeded / padding)
  __shared__ uint16_t s_tok[TMAX];         // tokens of this workgroup's slots, grouped, eviction order
  __shared__ int s_cnt[AGG_SLOTS];
  __shared__ int s_off[AGG_SLOTS + 1];       // local slot q = group + 16 * pass
  // the workgroup's tokens in list order, [position][K, V][D] KV dtype, when they fit
  __shared__ __attribute__((aligned(16))) uint8_t s_tk[AGG_TOK_BYTES];
  // EMA centres: the unit's codebooks [K, V][G][CMAX][DP] for the residual
  // codes, and the code of every (token, K/V, subspace) of the workgroup
  __shared__ __attribute__((aligned(16))) float s_cb[EMA ? 2 * G * CMAX * DP : 4];
  __shared__ uint8_t s_code[EMA ? TMAX * 2 * G : 4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // same XCD placement as the screen (consecutive logical blocks share an
  // XCD), so the unit's assignments and evicted tokens come from its L2
  const int nblk = (int)gridDim.x, per = nblk >> 3, bid = (int)blockIdx.x;
  const int lb = bid < per * 8 ? (bid & 7) * per + (bid >> 3) : bid;
  const int wgi = lb % wg_per_unit;
  const int bu = lb / wg_per_unit;
  const int b = bu / dm.units, u = bu % dm.units;
  const int N = dm.T;
  const int nseed = fb.nseed[b];
  const int kact = fb.nact[b] + nseed;
  const int k0 = wgi * AGG_SLOTS;
  if (nseed >= N || k0 >= kact) return;  // uniform
  const size_t unit = (size_t)fb.sid[b] * dm.units + u;
  const bool pq = (dm.flags & PROTOKV_FLAG_PQ) != 0 && !fb.warm[b];  // warm-up folds count no codes
  const size_t fbase = ((unit * (dm.W + 1) + fb.slot[b]) * N) * (size_t)D;
  const unsigned long long below = (1ull << lane) - 1ull;
  const int N64 = (N + 63) & ~63;

  for (int j = tid; j < N64; j += 256)
    s_asg[j] = (j >= nseed && j < N) ? (uint16_t)ws.assign[unit * N + j] : NO_SLOT;
  __syncthreads();
  // wave w sweeps for the local slots of its lane groups: q = 4 w + g + 16 p
  // (slot k0 + q), g = 0..3, p < NP
  int kw[NGW];
#pragma unroll
  for (int g = 0; g < NGW; ++g) {
    const int q = 4 * wave + (g & 3) + 16 * (g >> 2);
    kw[g] = (k0 + q < kact) ? k0 + q : -1;
  }
  int cw[NGW];
#pragma unroll
  for (int g = 0; g < NGW; ++g) cw[g] = 0;
  for (int c = 0; c < N64; c += 64) {
    const int a = s_asg[c + lane];
#pragma unroll
    for (int g = 0; g < NGW; ++g) cw[g] += __popcll(__ballot(a == kw[g]));
  }
  if (lane < NGW) {
    int v = cw[0];
#pragma unroll
    for (int g = 1; g < NGW; ++g) v = lane == g ? cw[g] : v;
    s_cnt[4 * wave + (lane & 3) + 16 * (lane >> 2)] = v;
  }
  __syncthreads();
  if (wave == 0) {
    // inclusive scan of the counts, entries lane and lane + 64
    int carry = 0;
#pragma unroll
    for (int h = 0; h < (AGG_SLOTS + 63) / 64; ++h) {
      const int e = h * 64 + lane;
      int incl = e < AGG_SLOTS ? s_cnt[e] : 0;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
      }
      if (e < AGG_SLOTS) s_off[e + 1] = carry + incl;
      carry += __shfl(incl, 63, 64);
    }
    if (lane == 0) s_off[0] = 0;
  }
  __syncthreads();
  if (s_off[AGG_SLOTS] == 0) return;  // uniform: none of these slots drew a token
  if (EMA && pq) {
    const float4* src = reinterpret_cast<const float4*>(ws.codebooks + unit * (2 * G * CMAX * DP));
    for (int x = tid; x < 2 * G * CMAX * DP / 4; x += 256) reinterpret_cast<float4*>(s_cb)[x] = src[x];
  }
  int ow[NGW];
#pragma unroll
  for (int g = 0; g < NGW; ++g) ow[g] = s_off[4 * wave + (g & 3) + 16 * (g >> 2)];
  for (int c = 0; c < N64; c += 64) {
    const int a = s_asg[c + lane];
#pragma unroll
    for (int g = 0; g < NGW; ++g) {
      const unsigned long long mk = __ballot(a == kw[g]);
      if (a == kw[g]) s_tok[ow[g] + __popcll(mk & below)] = (uint16_t)(c + lane);
      ow[g] += __popcll(mk);
    }
  }
  __syncthreads();

  const int gi = tid >> 4, il = tid & 15;
  const float eta = dm.eta, keep = 1.0f - dm.eta;
  constexpr int ES = FP32 ? 4 : 2;
  constexpr int TOKB = 2 * D * ES;             // bytes of one token's K and V
  constexpr int TPI = 1024 / TOKB;             // tokens per 1 KiB DMA instruction
  constexpr int CAP = AGG_TOK_BYTES / TOKB;
  // All of the workgroup's tokens go into LDS in one round of DMA loads
  // (instruction i moves list positions TPI i ..: lane = (position, K/V,
  // 16-byte part)), beside the first slot's row loads; a workgroup with more
  // tokens than fit reads them from global memory TOK_BATCH at a time.
  const int ntok = s_off[AGG_SLOTS];
  const bool staged = ntok <= CAP;  // uniform
  if (staged) {
    const int ninstr = (ntok + TPI - 1) / TPI;
    for (int i = wave; i < ninstr; i += 4) {
      const int pos = min(TPI * i + (FP32 ? 0 : (lane >> 5)), ntok - 1);
      const int kvs = FP32 ? (lane >> 5) : ((lane >> 4) & 1);
      const int part = FP32 ? (lane & 31) : (lane & 15);
      const uint8_t* src = (kvs ? ws.ring_v : ws.ring_k) + (fbase + (size_t)s_tok[pos] * D) * ES + part * 16;
      lds_dma16(src, s_tk + i * 1024);
    }
  }
  // the group's first touched slot's row (loads in flight with the
  // tokens'); each later touched slot's row is loaded while the one before
  // it absorbs its tokens
  float sk[8], sv[8], qk[8], qv[8];
  float nk[8], nv[8], nqk[8], nqv[8];
  RowMeta m, nm;
  auto load_row = [&](int q, float (&a)[8], float (&b)[8], float (&c)[8], float (&d)[8], RowMeta& mm) {
    const uint8_t* row = ws.bank + (unit * dm.K + k0 + q) * ROW;
    ld8f(row + ROW_SUMK + il * 32, a);
    ld8f(row + ROW_SUMV + il * 32, b);
    ld8f(row + ROW_SQK + il * 32, c);
    ld8f(row + ROW_SQV + il * 32, d);
    mm = *reinterpret_cast<const RowMeta*>(row + ROW_META);
  };
  // next pass >= p with tokens for this group (NP if none)
  auto next_pass = [&](int p) {
    while (p < NP && s_off[gi + 16 * p + 1] == s_off[gi + 16 * p]) ++p;
    return p;
  };
  const float ak = dm.alpha, av = dm.beta, a1k = 1.0f - dm.alpha, a1v = 1.0f - dm.beta;
  int pnext = next_pass(0);
  if (pnext < NP) load_row(gi + 16 * pnext, sk, sv, qk, qv, m);
  if (staged) {
    wait_vm<0>();  // this wave's token loads (and its row loads) have landed
    __syncthreads();
  }
  for (int pass = pnext; pass < NP; pass = pnext) {  // uniform per lane group; no barrier below
    const int q = gi + 16 * pass;
    const int t0 = s_off[q], t1 = s_off[q + 1];
    const int k = k0 + q;
    const size_t si = unit * dm.K + k;
    uint8_t* row = ws.bank + si * ROW;
    pnext = next_pass(pass + 1);
    if (NP > 2 && pnext < NP) load_row(gi + 16 * pnext, nk, nv, nqk, nqv, nm);
    for (int tb = t0; tb < t1; tb += TOK_BATCH) {  // uniform per lane group
      // a batch's loads all in flight together (indices clamped into the list)
      int jb[TOK_BATCH];
      Raw8<FP32> kb[TOK_BATCH], vb[TOK_BATCH];
#pragma unroll
      for (int e = 0; e < TOK_BATCH; ++e) {
        const int pos = min(tb + e, t1 - 1);
        jb[e] = s_tok[pos];
        if (staged) {
          const uint4* pk = reinterpret_cast<const uint4*>(s_tk + pos * TOKB + il * 8 * ES);
          const uint4* pv = reinterpret_cast<const uint4*>(s_tk + pos * TOKB + D * ES + il * 8 * ES);
#pragma unroll
          for (int w = 0; w < (FP32 ? 2 : 1); ++w) {
            kb[e].w[w] = pk[w];
            vb[e].w[w] = pv[w];
          }
        } else {
          load8<FP32>(ws.ring_k, fbase + (size_t)jb[e] * D + 8 * il, kb[e]);
          load8<FP32>(ws.ring_v, fbase + (size_t)jb[e] * D + 8 * il, vb[e]);
        }
      }
#pragma unroll
      for (int e = 0; e < TOK_BATCH; ++e) {
        if (tb + e < t1) {
          const int jj = jb[e];
          if (EMA) {
            // c <- (1 - alpha) c + alpha K, p likewise with beta; residuals
            // against the updated centres to the workspace (coded below)
            float rk[8], rv[8];
#pragma unroll
            for (int d = 0; d < 8; ++d) {
              const float xk = raw_at<FP32>(kb[e], d), xv = raw_at<FP32>(vb[e], d);
              sk[d] = a1k * sk[d] + ak * xk;
              sv[d] = a1v * sv[d] + av * xv;
              qk[d] = qk[d] + xk * xk;
              qv[d] = qv[d] + xv * xv;
              rk[d] = xk - sk[d];
              rv[d] = xv - sv[d];
            }
            if (pq) {
              float* rr = ws.ema_res + ((unit * N + jj) * 2) * (size_t)D + 8 * il;
              // read back by this workgroup below: ordinary stores
              *reinterpret_cast<float4*>(rr) = make_float4(rk[0], rk[1], rk[2], rk[3]);
              *reinterpret_cast<float4*>(rr + 4) = make_float4(rk[4], rk[5], rk[6], rk[7]);
              *reinterpret_cast<float4*>(rr + D) = make_float4(rv[0], rv[1], rv[2], rv[3]);
              *reinterpret_cast<float4*>(rr + D + 4) = make_float4(rv[4], rv[5], rv[6], rv[7]);
              m.n_res += 1;
            }
          } else {
#pragma unroll
            for (int d = 0; d < 8; ++d) {
              const float xk = raw_at<FP32>(kb[e], d), xv = raw_at<FP32>(vb[e], d);
              sk[d] = sk[d] + xk;
              sv[d] = sv[d] + xv;
              qk[d] = qk[d] + xk * xk;
              qv[d] = qv[d] + xv * xv;
            }
            if (pq) m.n_res += 1;
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
    }
    st8f(row + ROW_SUMK + il * 32, sk);
    st8f(row + ROW_SUMV + il * 32, sv);
    st8f(row + ROW_SQK + il * 32, qk);
    st8f(row + ROW_SQV + il * 32, qv);
    // the meta and the padding after it: one whole 64-byte sector
    if (il == 0) *reinterpret_cast<RowMeta*>(row + ROW_META) = m;
    if (il == 1) *reinterpret_cast<RowMeta*>(row + ROW_META + sizeof(RowMeta)) = RowMeta{};
    refresh_cache16(dm, sk, m, unit, k, ws, il);
    // per-slot count of folds that touched it (owned by this lane group: no atomics)
    if (il == 0) ws.touched[si] += 1u;
    if (pnext < NP) {
      if (NP > 2) {
#pragma unroll
        for (int d = 0; d < 8; ++d) {
          sk[d] = nk[d];
          sv[d] = nv[d];
          qk[d] = nqk[d];
          qv[d] = nqv[d];
        }
        m = nm;
      } else {
        load_row(gi + 16 * pnext, sk, sv, qk, qv, m);
      }
    }
  }
  if (EMA && pq) {
    // every (token, K/V, subspace) of the workgroup coded in parallel from
    // the residuals written above: the float32 sequential distance over the
    // subspace's dims, ascending, ties to the lower codeword.  Tasks run
    // token-fastest, so a wave's lanes share one codebook (broadcast reads).
    __syncthreads();
    for (int task = tid; task < ntok * 2 * G; task += 256) {
      const int pos = task % ntok, sg = task / ntok, side = sg / G, g = sg % G;
      const float* rr = ws.ema_res + ((unit * N + s_tok[pos]) * 2 + side) * (size_t)D + g * DP;
      float x[DP];
#pragma unroll
      for (int q = 0; q < DP / 4; ++q) {
        const float4 v = reinterpret_cast<const float4*>(rr)[q];
        x[4 * q] = v.x; x[4 * q + 1] = v.y; x[4 * q + 2] = v.z; x[4 * q + 3] = v.w;
      }
      const float* cw = s_cb + (side * G + g) * CMAX * DP;
      float best = INFINITY;
      int code = 0;
      for (int c = 0; c < dm.C; ++c) {
        float acc = 0.f;
#pragma unroll
        for (int d = 0; d < DP; ++d) {
          const float df = x[d] - cw[c * DP + d];
          acc = acc + df * df;
        }
        if (acc < best) {
          best = acc;
          code = c;
        }
      }
      s_code[pos * 2 * G + side * G + g] = (uint8_t)code;
    }
    __syncthreads();
    // each group adds its slots' codes to their histograms: lane il holds
    // bins H[il / 2][8 (il % 2) ..] of K and of V
    for (int pass = 0; pass < NP; ++pass) {
      const int q = gi + 16 * pass;
      const int t0 = s_off[q], t1 = s_off[q + 1];
      if (t1 == t0) continue;
      uint8_t* row = ws.bank + (unit * dm.K + k0 + q) * ROW;
      uint4* phk = reinterpret_cast<uint4*>(row + ROW_HK + il * 32);
      uint4* phv = reinterpret_cast<uint4*>(row + ROW_HV + il * 32);
      uint4 h0 = phk[0], h1 = phk[1], v0 = phv[0], v1 = phv[1];
      const int sg = il >> 1, base = 8 * (il & 1);
      for (int pos = t0; pos < t1; ++pos) {
        const int zk = (int)s_code[pos * 2 * G + sg] - base, zv = (int)s_code[pos * 2 * G + G + sg] - base;
        h0.x += zk == 0; h0.y += zk == 1; h0.z += zk == 2; h0.w += zk == 3;
        h1.x += zk == 4; h1.y += zk == 5; h1.z += zk == 6; h1.w += zk == 7;
        v0.x += zv == 0; v0.y += zv == 1; v0.z += zv == 2; v0.w += zv == 3;
        v1.x += zv == 4; v1.y += zv == 5; v1.z += zv == 6; v1.w += zv == 7;
      }
      phk[0] = h0;
      phk[1] = h1;
      phv[0] = v0;
      phv[1] = v1;
    }
  }
}

// ---------------------------------------------------------------------------
// Aggregation over the touched slots only (running means, K <= AGC_KMAX).
// A fold touches a fraction of the K slots (about 100 of 512 on a 7B-shaped
// stream), so workgroups over fixed ranges of slots spend most of their lane
// groups on slots without tokens.  Here each of the P workgroups of a unit
// buckets the unit's evicted tokens by slot in LDS (per-slot counts by LDS
// atomics, one exclusive scan that also numbers the touched slots, a scatter
// and a stable re-ranking, so every slot's tokens are in eviction order),
// then its 16 lane groups take touched slots gi + 16 (p + P r): the row's
// four sums go to registers (lane il: dims [8 il, 8 il + 8)), the slot's
// tokens are absorbed in order TOK_BATCH at a time with their loads in
// flight, the row and the slot's screening copy are written back, and the
// next touched slot's row is loaded before the current one's stores.  The
// arithmetic is k_aggregate's: the same float32 operation sequence per slot.
// ---------------------------------------------------------------------------
constexpr int AGC_KMAX = 4096;  // slot counters held in LDS

template <int FP32>
__global__ __launch_bounds__(256, 4) void k_aggregate_c(Dims dm, Workspace ws, FoldBatch fb, int wg_per_unit) {
  // per slot: token count | touched flag << 16, then the exclusive prefix of
  // both (list offset | touched index << 16); entry K holds the totals
  __shared__ uint32_t s_cnt[AGC_KMAX + 1];
  __shared__ uint16_t s_asg[TMAX];     // slot of token j
  __shared__ uint16_t s_pos[TMAX];     // arrival index of token j among its slot's tokens
  __shared__ uint16_t s_list[TMAX];    // tokens grouped by slot, arrival order
  __shared__ uint16_t s_tok[TMAX];     // the same groups in eviction order
  __shared__ uint16_t s_tslot[TMAX];   // touched slots, ascending
  __shared__ uint16_t s_tstart[TMAX + 1];
  __shared__ uint32_t s_wsum[4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nblk = (int)gridDim.x, per = nblk >> 3, bid = (int)blockIdx.x;
  const int lb = bid < per * 8 ? (bid & 7) * per + (bid >> 3) : bid;
  const int wgi = lb % wg_per_unit;
  const int bu = lb / wg_per_unit;
  const int b = bu / dm.units, u = bu % dm.units;
  const int N = dm.T, K = dm.K;
  const int nseed = fb.nseed[b];
  if (nseed >= N) return;  // uniform
  const size_t unit = (size_t)fb.sid[b] * dm.units + u;
  const bool pq = (dm.flags & PROTOKV_FLAG_PQ) != 0 && !fb.warm[b];  // warm-up folds count no codes
  const size_t fbase = ((unit * (dm.W + 1) + fb.slot[b]) * N) * (size_t)D;

  // 1. counts per slot
  for (int k = tid; k <= K; k += 256) s_cnt[k] = 0u;
  __syncthreads();
  for (int j = nseed + tid; j < N; j += 256) {
    const int k = ws.assign[unit * N + j];
    s_asg[j] = (uint16_t)k;
    s_pos[j] = (uint16_t)atomicAdd(&s_cnt[k], 1u);
  }
  __syncthreads();
  // 2. exclusive scan of (count | touched << 16): thread tid owns slots
  // [tid E, tid E + E); counts stay below 2^16, so the two fields add apart
  const int E = (K + 255) >> 8;
  const int ka = min(K, tid * E), kb = min(K, ka + E);
  uint32_t own = 0u;
  for (int k = ka; k < kb; ++k) {
    const uint32_t c = s_cnt[k];
    own += c + (c ? 0x10000u : 0u);
  }
  uint32_t incl = own;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  if (lane == 63) s_wsum[wave] = incl;
  __syncthreads();
  uint32_t base = 0u;
  for (int w = 0; w < wave; ++w) base += s_wsum[w];
  uint32_t run = base + incl - own;
  for (int k = ka; k < kb; ++k) {
    const uint32_t c = s_cnt[k];
    s_cnt[k] = run;
    if (c) {
      s_tslot[run >> 16] = (uint16_t)k;
      s_tstart[run >> 16] = (uint16_t)(run & 0xFFFFu);
    }
    run += c + (c ? 0x10000u : 0u);
  }
  const uint32_t total = s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3];
  const int ntouched = (int)(total >> 16), ntok = (int)(total & 0xFFFFu);
  if (tid == 0) {
    s_cnt[K] = total;
    s_tstart[ntouched] = (uint16_t)ntok;
  }
  __syncthreads();
  // 3. scatter (arrival order), then each token's rank among its slot's
  // tokens by index: the eviction order
  for (int j = nseed + tid; j < N; j += 256) s_list[(s_cnt[s_asg[j]] & 0xFFFFu) + s_pos[j]] = (uint16_t)j;
  __syncthreads();
  for (int j = nseed + tid; j < N; j += 256) {
    const int k = s_asg[j];
    const int a = (int)(s_cnt[k] & 0xFFFFu), e = (int)(s_cnt[k + 1] & 0xFFFFu);
    int rank = 0;
    for (int m = a; m < e; ++m) rank += s_list[m] < j ? 1 : 0;
    s_tok[a + rank] = (uint16_t)j;
  }
  __syncthreads();

  // 4. the lane groups' touched slots
  const int gi = tid >> 4, il = tid & 15;
  const int step = 16 * wg_per_unit;
  int ti = gi + 16 * wgi;
  if (ti >= ntouched) return;  // uniform per lane group; no barrier below
  const float eta = dm.eta, keep = 1.0f - dm.eta;
  float sk[8], sv[8], qk[8], qv[8];
  float nk[8], nv[8], nqk[8], nqv[8];
  RowMeta m, nm;
  auto load_row = [&](int k, float (&a)[8], float (&b2)[8], float (&c)[8], float (&d)[8], RowMeta& mm) {
    const uint8_t* row = ws.bank + (unit * K + k) * ROW;
    ld8f(row + ROW_SUMK + il * 32, a);
    ld8f(row + ROW_SUMV + il * 32, b2);
    ld8f(row + ROW_SQK + il * 32, c);
    ld8f(row + ROW_SQV + il * 32, d);
    mm = *reinterpret_cast<const RowMeta*>(row + ROW_META);
  };
  load_row(s_tslot[ti], sk, sv, qk, qv, m);
  for (; ti < ntouched; ti += step) {
    const int k = s_tslot[ti];
    const int t0 = s_tstart[ti], t1 = s_tstart[ti + 1];
    const size_t si = unit * K + k;
    uint8_t* row = ws.bank + si * ROW;
    const int tn = ti + step;
    for (int tb = t0; tb < t1; tb += TOK_BATCH) {
      int jb[TOK_BATCH];
      Raw8<FP32> kb2[TOK_BATCH], vb2[TOK_BATCH];
#pragma unroll
      for (int e = 0; e < TOK_BATCH; ++e) {
        jb[e] = s_tok[min(tb + e, t1 - 1)];
        load8<FP32>(ws.ring_k, fbase + (size_t)jb[e] * D + 8 * il, kb2[e]);
        load8<FP32>(ws.ring_v, fbase + (size_t)jb[e] * D + 8 * il, vb2[e]);
      }
#pragma unroll
      for (int e = 0; e < TOK_BATCH; ++e) {
        if (tb + e < t1) {
          const int jj = jb[e];
#pragma unroll
          for (int d = 0; d < 8; ++d) {
            const float xk = raw_at<FP32>(kb2[e], d), xv = raw_at<FP32>(vb2[e], d);
            sk[d] = sk[d] + xk;
            sv[d] = sv[d] + xv;
            qk[d] = qk[d] + xk * xk;
            qv[d] = qv[d] + xv * xv;
          }
          if (pq) m.n_res += 1;
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
    }
    // the next touched slot's row in flight before this one's stores
    if (tn < ntouched) load_row(s_tslot[tn], nk, nv, nqk, nqv, nm);
    st8f(row + ROW_SUMK + il * 32, sk);
    st8f(row + ROW_SUMV + il * 32, sv);
    st8f(row + ROW_SQK + il * 32, qk);
    st8f(row + ROW_SQV + il * 32, qv);
    // the meta and the padding after it: one whole 64-byte sector
    if (il == 0) *reinterpret_cast<RowMeta*>(row + ROW_META) = m;
    if (il == 1) *reinterpret_cast<RowMeta*>(row + ROW_META + sizeof(RowMeta)) = RowMeta{};
    refresh_cache16(dm, sk, m, unit, k, ws, il);
    if (il == 0) ws.touched[si] += 1u;
    if (tn < ntouched) {
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        sk[d] = nk[d];
        sv[d] = nv[d];
        qk[d] = nqk[d];
        qv[d] = nqv[d];
      }
      m = nm;
    }
  }
}

hipError_t launch_aggregate(const Dims& dm, const Workspace& ws, const FoldBatch& fb, hipStream_t st) {
  const bool ema = (dm.flags & PROTOKV_FLAG_EMA_CENTRES) != 0;
  if (!ema && dm.K <= AGC_KMAX) {
    // touched slots only: P workgroups per unit, enough to put about 2048
    // workgroups in flight, at most one per 16 slots a fold can touch
    const int units = fb.n * dm.units;
    const int pmax = (std::min(dm.T, dm.K) + 15) / 16;
    const int P = std::max(1, std::min(pmax, (2048 + units - 1) / units));
    dim3 grid(units * P);
    using KFn = void (*)(Dims, Workspace, FoldBatch, int);
    const KFn fn = dm.kv_fp32 ? k_aggregate_c<1> : k_aggregate_c<0>;
    hipLaunchKernelGGL(fn, grid, dim3(256), 0, st, dm, ws, fb, P);
    return hipGetLastError();
  }
  // running means: AGG_NP slots per lane group (16 AGG_NP per workgroup);
  // EMA centres code their residuals in the workgroup: two per group
  constexpr int NPM = AGG_NP;
  const int slots = ema ? 32 : 16 * NPM;
  const int wpu = (dm.K + slots - 1) / slots;
  dim3 grid(fb.n * dm.units * wpu);
  using KFn = void (*)(Dims, Workspace, FoldBatch, int);
  const KFn fn = dm.kv_fp32 ? (ema ? k_aggregate<1, 1, 2> : k_aggregate<1, 0, NPM>)
                            : (ema ? k_aggregate<0, 1, 2> : k_aggregate<0, 0, NPM>);
  hipLaunchKernelGGL(fn, grid, dim3(256), 0, st, dm, ws, fb, wpu);
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Prototype maintenance (Alg. "Prototype Maintenance") after a fold, over the
// A = nact + nseed seeded slots of one (stream, unit); workgroup of MT_WAVES
// waves.
//  1. Aging (threads over slots, then over 16-byte pieces): an idle slot gets
//     n' = floor((1 - gamma) n) in float64 and its sums and squared sums are
//     scaled by float32(n') / float32(n); the first FD dims of every slot's
//     key and value centres float32(sum / n) go to LDS (FD = 16, 8 or 4 as
//     K grows).
//  2. Merging, i ascending: i absorbs every later j whose key and value
//     centres are closer than eps_k and eps_v.  A squared distance is the
//     float64 terms (c_i[d] - c_j[d])^2 summed in a fixed tree: dims 2L and
//     2L + 1 first, then the 64 pair sums by halves of L (bit 5 first, bit 0
//     last).  Rows go in blocks of mt_block(K); per block:
//     a. a filter on the LDS dims over every pair i < j with i in the block:
//        the partial sum of squares over the filter dims is a lower bound of
//        the full one; the waves form it for 32 x 32 pair tiles in the Gram
//        form on MFMA (bound below) and list the pairs whose key and value
//        partials may be below eps_k^2 and eps_v^2 (1e-4 relative slack for
//        the float64 rounding of the exact sums, plus the Gram bound);
//     b. groups of 16 lanes test the listed pairs exactly and mark those
//        that merge in a bitmask [block rows][K];
//     c. wave 0 walks the marked rows: while i's centre has not moved, its
//        partners are the marked j still holding mass (neither centre has
//        changed since: a later slot only loses its mass to an earlier row);
//        after i's first merge, and for rows whose pairs overflowed the
//        list, it runs the filter as float32 sums of squares, 64 candidates
//        at a time, and tests each candidate exactly (64 lanes, same tree).
//     i absorbs j: sums, squared sums, histograms, n and n_res add, mu the
//     mass-weighted mean; i's centre (registers and LDS) moves at once.
//  3. Recycling (waves over a worklist): the empty slots, in ascending
//     order, take the near window's tokens, newest frame first, raster order.
//  4. The screening copies of aged and absorbing slots are rewritten
//     (recycled slots are rewritten as they are seeded).
// ---------------------------------------------------------------------------
constexpr int MT_PAIRS = 4096;  // filter pairs listed per block
constexpr int MT_THREADS = 512, MT_WAVES = MT_THREADS / 64;
// Gram form of the filter: P = |a|^2 + |b|^2 - 2 a.b over the filter dims of
// two float32 centres, a.b on MFMA from hi + lo bf16 splits (hi*hi + hi*lo +
// lo*hi, float32 accumulation).  The split leaves at most 2^-16 |x| per
// component, the dropped lo*lo term and the accumulation add at most 2^-17.4
// sum |a_d b_d|, so |a.b - computed| <= 2^-14.1 |a| |b|; with the float32
// norms, |P - (|a|^2 + |b|^2 - 2 computed)| <= 2^-13.9 S, S = |a|^2 + |b|^2.
// A pair is kept when rho_i + (rho_j + thr) - 2 computed <= 0 with the row
// terms rho = (1 - M) |x|^2 - thr (M = MT_GRAM_MARGIN): the test's own
// roundings stay below 2^-20 S + 2^-21 thr, so every pair with P below thr
// is kept.
constexpr float MT_GRAM_MARGIN = 0x1p-12f;

__host__ __device__ inline int mt_fd(int K) { return K <= 512 ? 16 : (K <= 1024 ? 8 : 4); }
__host__ __device__ inline int mt_w32(int K) { return (K + 31) / 32; }
// rows per block (a multiple of 32 below K): the bitmask holds at most 32 KiB
__host__ __device__ inline int mt_block(int K) {
  const int r = 8192 / mt_w32(K);
  return r < K ? (r & ~31) : K;
}
__host__ __device__ inline size_t mt_base_bytes(int K) {
  return (((size_t)K * (2 * mt_fd(K) * 4 + 4 + 4 + 2 + 1) + (size_t)cap32(K) * 8) + 15) & ~(size_t)15;
}
// dynamic LDS of k_maintain for capacity K: filter dims, masses, aging
// ratios, Gram row terms (key, value; K32 entries each), idle list /
// recycling ranks, stale flags | bitmask, marked-row flags, overflow flags |
// pair list (then the recycling and refresh worklist)
__host__ __device__ inline size_t mt_lds_bytes(int K) {
  const size_t R = (size_t)mt_block(K);
  return mt_base_bytes(K) + (R * mt_w32(K) + 2 * ((R + 31) / 32)) * 4 + (size_t)MT_PAIRS * 4;
}

// Squared key and value distances of two slots by a 16-lane group: lane m
// holds dims 2L, 2L + 1 for L = m + 16 r (r = 0 .. 3), so the first two tree
// levels (bits 5 and 4 of L) are in registers and the last four are lane
// exchanges within the group.
__device__ __forceinline__ void mt_dist16(const float2 (&ak)[4], const float2 (&av)[4], const float2 (&bk)[4],
                                          const float2 (&bv)[4], double& dk, double& dv) {
  double sk[4], sv[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const double ax = (double)ak[r].x - (double)bk[r].x, ay = (double)ak[r].y - (double)bk[r].y;
    const double bx = (double)av[r].x - (double)bv[r].x, by = (double)av[r].y - (double)bv[r].y;
    sk[r] = ax * ax + ay * ay;
    sv[r] = bx * bx + by * by;
  }
  dk = (sk[0] + sk[2]) + (sk[1] + sk[3]);
  dv = (sv[0] + sv[2]) + (sv[1] + sv[3]);
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) {
    dk = dk + __shfl_xor(dk, o, 64);
    dv = dv + __shfl_xor(dv, o, 64);
  }
}

template <int FP32, int FD>
__global__ __launch_bounds__(MT_THREADS) void k_maintain(Dims dm, Workspace ws, FoldBatch fb) {
  extern __shared__ __attribute__((aligned(16))) uint8_t s_dyn[];
  __shared__ int s_cnt[3];  // aged, merged, recycled
  __shared__ int s_np;      // pairs that passed the filter in this block
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int b = blockIdx.x / dm.units, u = blockIdx.x % dm.units;
  const int A = fb.nact[b] + fb.nseed[b];
  if (A <= 0) return;  // uniform
  const int t = fb.t[b];
  const int T = dm.T;
  const size_t unit = (size_t)fb.sid[b] * dm.units + u;
  uint8_t* rows = ws.bank + unit * dm.K * ROW;
  float* s_c16 = reinterpret_cast<float*>(s_dyn);  // [2 FD][K]: key dims, then value dims, dim-major
  // Gram row terms (1 - M) |filter dims|^2 - thr of key and value, +inf for
  // empty slots and from A up to K32 (16-byte aligned for b128 reads)
  float* s_rhk = s_c16 + (size_t)dm.K * 2 * FD;
  float* s_rhv = s_rhk + cap32(dm.K);
  uint32_t* s_n = reinterpret_cast<uint32_t*>(s_rhv + cap32(dm.K));  // [A] current mass
  float* s_r = reinterpret_cast<float*>(s_n + dm.K);                  // [A] aging ratio
  uint16_t* s_rk = reinterpret_cast<uint16_t*>(s_r + dm.K);          // [A] idle slots, later recycling ranks
  uint8_t* s_dirty = reinterpret_cast<uint8_t*>(s_rk + dm.K);        // [A] screening copy stale
  const int W32 = mt_w32(dm.K), R = mt_block(dm.K), RW = (R + 31) / 32;
  uint32_t* s_adj = reinterpret_cast<uint32_t*>(s_dyn + mt_base_bytes(dm.K));  // [R][W32]: (i, j) merges
  uint32_t* s_rf = s_adj + (size_t)R * W32;                                    // [RW]: row has a mark
  uint32_t* s_ov = s_rf + RW;                                                  // [RW]: row's pairs overflowed
  uint32_t* s_pairs = s_ov + RW;                                               // [MT_PAIRS]: i << 16 | j
  const unsigned long long below = (1ull << lane) - 1ull;
  if (tid < 3) s_cnt[tid] = 0;
  __syncthreads();

  const double ek2 = dm.eps_k * dm.eps_k, ev2 = dm.eps_v * dm.eps_v;
  const float fk2 = (float)(ek2 * (1.0 + 1e-4)), fv2 = (float)(ev2 * (1.0 + 1e-4));
  // 1a. aging, one thread per slot (its mass, tau and leading FD key and
  // value sums loaded together): mass after aging, idle slots listed, the
  // filter dims of the centres after aging and the Gram row terms
  // (1 - M) |filter dims|^2 - thr, +inf for empty slots and past A
  {
    constexpr int QC = FD / 4;  // 16-byte chunks per side
    for (int k = tid; k < cap32(dm.K); k += MT_THREADS) {
      float rk = INFINITY, rv = INFINITY;
      if (k < A) {
        uint8_t* row = rows + (size_t)k * ROW;
        uint32_t* mp = reinterpret_cast<uint32_t*>(row + ROW_META);
        float4 f[2][QC];
#pragma unroll
        for (int q = 0; q < QC; ++q) {
          f[0][q] = *reinterpret_cast<const float4*>(row + ROW_SUMK + 16 * q);
          f[1][q] = *reinterpret_cast<const float4*>(row + ROW_SUMV + 16 * q);
        }
        const uint32_t n = mp[0];                         // RowMeta::n
        const int32_t tau = static_cast<int32_t>(mp[7]);  // RowMeta::tau
        const bool idle = (t - tau / T) > dm.t_idle;
        uint32_t n2 = n;
        float r = 1.f;
        if (idle) {
          n2 = (uint32_t)floor((1.0 - dm.gamma) * (double)n);
          r = (float)n2 / (float)n;
          mp[0] = n2;
          s_rk[atomicAdd(&s_cnt[0], 1)] = (uint16_t)k;
        }
        s_n[k] = n2;
        s_r[k] = r;
        s_dirty[k] = idle ? 1 : 0;
        const float nf = (float)n2;
        float nrm[2] = {0.f, 0.f};
#pragma unroll
        for (int side = 0; side < 2; ++side)
#pragma unroll
          for (int q = 0; q < QC; ++q) {
            const float fv[4] = {f[side][q].x, f[side][q].y, f[side][q].z, f[side][q].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float y = idle ? fv[e] * r : fv[e];
              const float c = n2 > 0 ? y / nf : 0.f;
              s_c16[(side * FD + 4 * q + e) * dm.K + k] = c;
              nrm[side] = fmaf(c, c, nrm[side]);
            }
          }
        if (n2 > 0) {
          rk = (1.f - MT_GRAM_MARGIN) * nrm[0] - fk2;
          rv = (1.f - MT_GRAM_MARGIN) * nrm[1] - fv2;
        }
      }
      s_rhk[k] = rk;
      s_rhv[k] = rv;
    }
  }
  __syncthreads();
  const int nidle = s_cnt[0];
  // 1c. idle slots: sums and squared sums scaled by float32(n') / float32(n),
  // one thread per 16 bytes
  for (int x = tid; x < nidle * 128; x += MT_THREADS) {
    const int k = s_rk[x >> 7];
    float4* pf = reinterpret_cast<float4*>(rows + (size_t)k * ROW + ROW_SUMK) + (x & 127);
    const float r = s_r[k];
    const float4 f = *pf;
    *pf = make_float4(f.x * r, f.y * r, f.z * r, f.w * r);
  }

  int nmerged = 0;  // wave 0
  for (int r0 = 0; r0 < A; r0 += R) {  // uniform
    const int r1 = min(A, r0 + R);
    for (int x = tid; x < R * W32 + 2 * RW; x += MT_THREADS) s_adj[x] = 0u;
    if (tid == 0) s_np = 0;
    __syncthreads();

    // 2a. filter on MFMA: 32 x 32 tiles (rows ib of the block, columns jb >=
    // ib) of the Gram matrices of the filter dims, tiles t = wave, wave + W,
    // ... in row-major order; the pairs that pass are listed
    {
      const int col = lane & 31, half = lane >> 5;
      const int nb = (A + 31) >> 5;
      // operand of slot s: dims 8 half .. 8 half + 7 of one side, hi + lo
      auto operand = [&](int s, int side, bf16x8& h, bf16x8& l) {
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int d = 8 * half + e;
          v[e] = d < FD ? s_c16[(side * FD + d) * dm.K + s] : 0.f;
        }
        split8(v, h, l);
      };
      int tc = 0;
      for (int ib = r0 >> 5; ib < ((r1 + 31) >> 5); ++ib) {  // uniform
        const int jb0 = ib + ((wave - tc) % MT_WAVES + MT_WAVES) % MT_WAVES;
        tc += nb - ib;
        if (jb0 >= nb) continue;
        bf16x8 akh, akl, avh, avl;
        {
          const int si = min(ib * 32 + col, A - 1);
          operand(si, 0, akh, akl);
          operand(si, 1, avh, avl);
        }
        // accumulator element rr is row (rr / 4) * 8 + half * 4 + rr % 4:
        // its row terms, +inf past the block
        float rhk[16], rhv[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int i0 = ib * 32 + q * 8 + half * 4;
          const float4 xk = *reinterpret_cast<const float4*>(s_rhk + i0);
          const float4 xv = *reinterpret_cast<const float4*>(s_rhv + i0);
          const float ek[4] = {xk.x, xk.y, xk.z, xk.w}, ev[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            rhk[4 * q + r] = i0 + r < r1 ? ek[r] : INFINITY;
            rhv[4 * q + r] = i0 + r < r1 ? ev[r] : INFINITY;
          }
        }
        for (int jb = jb0; jb < nb; jb += MT_WAVES) {  // uniform
          const int j = jb * 32 + col, jc = min(j, A - 1);
          bf16x8 bkh, bkl, bvh, bvl;
          operand(jc, 0, bkh, bkl);
          operand(jc, 1, bvh, bvl);
          // column terms (1 - M) |b|^2 = row term + thr (+inf past A or empty)
          const float gck = s_rhk[j] + fk2, gcv = s_rhv[j] + fv2;
          const bool diag = jb == ib;
          f32x16 gk = {}, gv = {};
          gk = __builtin_amdgcn_mfma_f32_32x32x16_bf16(akh, bkh, gk, 0, 0, 0);
          gv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(avh, bvh, gv, 0, 0, 0);
          gk = __builtin_amdgcn_mfma_f32_32x32x16_bf16(akh, bkl, gk, 0, 0, 0);
          gv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(avh, bvl, gv, 0, 0, 0);
          gk = __builtin_amdgcn_mfma_f32_32x32x16_bf16(akl, bkh, gk, 0, 0, 0);
          gv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(avl, bvh, gv, 0, 0, 0);
          // pair (i, j) passes when max(row + column - 2 G) over key and
          // value is <= 0 (and i < j on the diagonal tile)
          float e[16], emin = INFINITY;
#pragma unroll
          for (int rr = 0; rr < 16; ++rr) {
            const int m = (rr >> 2) * 8 + half * 4 + (rr & 3);
            const float tk = fmaf(-2.f, gk[rr], rhk[rr] + gck);
            const float tv = fmaf(-2.f, gv[rr], rhv[rr] + gcv);
            e[rr] = (diag && m >= col) ? INFINITY : fmaxf(tk, tv);
            emin = fminf(emin, e[rr]);
          }
          if (__ballot(emin <= 0.f) == 0ull) continue;  // uniform
#pragma unroll
          for (int rr = 0; rr < 16; ++rr) {
            const bool pass = e[rr] <= 0.f;
            const unsigned long long bal = __ballot(pass);
            if (bal == 0ull) continue;  // uniform
            int base = 0;
            if (lane == 0) base = atomicAdd(&s_np, __popcll(bal));
            base = __shfl(base, 0, 64);
            const int pos = base + __popcll(bal & below);
            if (pass) {
              const int i = ib * 32 + (rr >> 2) * 8 + half * 4 + (rr & 3);
              if (pos < MT_PAIRS)
                s_pairs[pos] = ((uint32_t)i << 16) | (uint32_t)j;
              else
                atomicOr(&s_ov[(i - r0) >> 5], 1u << ((i - r0) & 31));
            }
          }
        }
      }
    }
    __syncthreads();

    // 2b. exact test of the listed pairs: groups of 16 lanes, two pairs
    // per group in flight
    {
      const int np = min(s_np, MT_PAIRS);
      constexpr int NG = MT_THREADS / 16;  // groups
      const int grp = tid >> 4, m = tid & 15;
      for (int p0 = grp; p0 < np; p0 += 2 * NG) {
        int pi[2], pj[2];
        bool ok[2];
        float2 ak[2][4], av[2][4], bk[2][4], bv[2][4];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int p = p0 + NG * h;
          const uint32_t e = p < np ? s_pairs[p] : 0u;
          pi[h] = (int)(e >> 16);
          pj[h] = (int)(e & 0xffffu);
          ok[h] = p < np;
          if (ok[h]) ok[h] = !((s_ov[(pi[h] - r0) >> 5] >> ((pi[h] - r0) & 31)) & 1u);  // overflowed: scanned
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            ak[h][r] = av[h][r] = bk[h][r] = bv[h][r] = make_float2(0.f, 0.f);
          }
          if (ok[h]) {
            const float2* xi = reinterpret_cast<const float2*>(rows + (size_t)pi[h] * ROW) + m;
            const float2* xj = reinterpret_cast<const float2*>(rows + (size_t)pj[h] * ROW) + m;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              ak[h][r] = xi[16 * r];
              av[h][r] = xi[64 + 16 * r];  // ROW_SUMV = 64 float2
              bk[h][r] = xj[16 * r];
              bv[h][r] = xj[64 + 16 * r];
            }
          }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const float ni = ok[h] ? (float)s_n[pi[h]] : 1.f, nj = ok[h] ? (float)s_n[pj[h]] : 1.f;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            ak[h][r] = make_float2(ak[h][r].x / ni, ak[h][r].y / ni);
            av[h][r] = make_float2(av[h][r].x / ni, av[h][r].y / ni);
            bk[h][r] = make_float2(bk[h][r].x / nj, bk[h][r].y / nj);
            bv[h][r] = make_float2(bv[h][r].x / nj, bv[h][r].y / nj);
          }
          double dk, dv;
          mt_dist16(ak[h], av[h], bk[h], bv[h], dk, dv);
          if (ok[h] && m == 0 && dk < ek2 && dv < ev2) {
            const int li = pi[h] - r0;
            atomicOr(&s_adj[li * W32 + (pj[h] >> 5)], 1u << (pj[h] & 31));
            atomicOr(&s_rf[li >> 5], 1u << (li & 31));
          }
        }
      }
    }
    __syncthreads();

    // 2c. merging (wave 0), marked rows ascending
    if (wave == 0) {
      for (int w = 0; w < (r1 - r0 + 31) / 32; ++w) {
        const uint32_t ovw = s_ov[w];
        uint32_t rword = s_rf[w] | ovw;
        while (rword != 0u) {  // uniform
          const int li = w * 32 + __ffs(rword) - 1;
          rword &= rword - 1u;
          const int i = r0 + li;
          if (s_n[i] == 0) continue;  // uniform
          uint8_t* rowi = rows + (size_t)i * ROW;
          // scan: pick candidates with the filter (after a merge, or when the
          // row's pairs overflowed the list); else from the bitmask
          bool scan = (ovw >> li) & 1u, have_ci = false;
          float2 cik = make_float2(0.f, 0.f), civ = make_float2(0.f, 0.f);  // dims 2l, 2l+1 of c_i, p_i
          int j0 = i + 1;
          while (j0 < A) {  // uniform
            int jj;
            if (!scan) {
              // lowest mark >= j0 of row i (lane l < W32 holds word l)
              uint32_t wv = lane < W32 ? s_adj[li * W32 + lane] : 0u;
              const int lo = j0 - lane * 32;
              if (lo > 0) wv = lo >= 32 ? 0u : (wv & ~((1u << lo) - 1u));
              const unsigned long long nz = __ballot(wv != 0u);
              if (nz == 0ull) break;
              const int wl = __ffsll((long long)nz) - 1;
              const uint32_t wsel = __shfl(wv, wl, 64);
              jj = wl * 32 + __ffs(wsel) - 1;
              if (s_n[jj] == 0) {  // merged away meanwhile
                j0 = jj + 1;
                continue;
              }
            } else {
              const int j = j0 + lane;
              bool pass = false;
              if (j < A && s_n[j] != 0) {
                float pk = 0.f, pv = 0.f;
#pragma unroll
                for (int d = 0; d < FD; ++d) {
                  const float dk = s_c16[d * dm.K + i] - s_c16[d * dm.K + j];
                  const float dv = s_c16[(FD + d) * dm.K + i] - s_c16[(FD + d) * dm.K + j];
                  pk = pk + dk * dk;
                  pv = pv + dv * dv;
                }
                pass = !(pk > fk2) && !(pv > fv2);
              }
              const unsigned long long bal = __ballot(pass);
              if (bal == 0ull) {
                j0 += 64;
                continue;
              }
              jj = j0 + __ffsll((long long)bal) - 1;
            }
            const uint8_t* rowj = rows + (size_t)jj * ROW;
            if (!have_ci) {
              const float ni = (float)s_n[i];
              const float2 sk = reinterpret_cast<const float2*>(rowi + ROW_SUMK)[lane];
              const float2 sv = reinterpret_cast<const float2*>(rowi + ROW_SUMV)[lane];
              cik = make_float2(sk.x / ni, sk.y / ni);
              civ = make_float2(sv.x / ni, sv.y / ni);
              have_ci = true;
            }
            const float nj = (float)s_n[jj];
            const float2 tk = reinterpret_cast<const float2*>(rowj + ROW_SUMK)[lane];
            const float2 tv = reinterpret_cast<const float2*>(rowj + ROW_SUMV)[lane];
            const float2 cjk = make_float2(tk.x / nj, tk.y / nj), cjv = make_float2(tv.x / nj, tv.y / nj);
            double dk, dv;
            {
              const double ax = (double)cik.x - (double)cjk.x, ay = (double)cik.y - (double)cjk.y;
              const double bx = (double)civ.x - (double)cjv.x, by = (double)civ.y - (double)cjv.y;
              dk = ax * ax + ay * ay;
              dv = bx * bx + by * by;
#pragma unroll
              for (int o = 32; o >= 1; o >>= 1) {
                dk = dk + __shfl_xor(dk, o, 64);
                dv = dv + __shfl_xor(dv, o, 64);
              }
            }
            if (dk < ek2 && dv < ev2) {  // uniform
              // i absorbs jj: lane l adds dims 2l, 2l+1 of the four sums and
              // histogram words 4l .. 4l+3 (H^K then H^V)
              float2 x[4];
#pragma unroll
              for (int a = 0; a < 4; ++a) {
                float2* pi = reinterpret_cast<float2*>(rowi + a * 512) + lane;
                const float2 xi = *pi, xj = reinterpret_cast<const float2*>(rowj + a * 512)[lane];
                x[a] = make_float2(xi.x + xj.x, xi.y + xj.y);
                *pi = x[a];
              }
              {
                uint4* hi = reinterpret_cast<uint4*>(rowi + ROW_HK) + lane;
                const uint4 h1 = *hi, h2 = reinterpret_cast<const uint4*>(rowj + ROW_HK)[lane];
                *hi = make_uint4(h1.x + h2.x, h1.y + h2.y, h1.z + h2.z, h1.w + h2.w);
              }
              const RowMeta mi = *reinterpret_cast<const RowMeta*>(rowi + ROW_META);
              const RowMeta mj = *reinterpret_cast<const RowMeta*>(rowj + ROW_META);
              const float wi = (float)mi.n, wj = (float)mj.n, wsum = wi + wj;
              RowMeta mn = mi;
              mn.mu_x = ((wi * mi.mu_x) + (wj * mj.mu_x)) / wsum;
              mn.mu_y = ((wi * mi.mu_y) + (wj * mj.mu_y)) / wsum;
              mn.n = mi.n + mj.n;
              mn.n_res = mi.n_res + mj.n_res;
              if (lane == 0) {
                *reinterpret_cast<RowMeta*>(rowi + ROW_META) = mn;
                *reinterpret_cast<uint32_t*>(const_cast<uint8_t*>(rowj) + ROW_META) = 0u;  // RowMeta::n
                s_n[i] = mn.n;
                s_n[jj] = 0u;
                s_dirty[i] = 1;
              }
              // i's centre moves
              const float nn = (float)mn.n;
              cik = make_float2(x[0].x / nn, x[0].y / nn);
              civ = make_float2(x[1].x / nn, x[1].y / nn);
              if (lane < FD / 2) {
                s_c16[(2 * lane) * dm.K + i] = cik.x;
                s_c16[(2 * lane + 1) * dm.K + i] = cik.y;
                s_c16[(FD + 2 * lane) * dm.K + i] = civ.x;
                s_c16[(FD + 2 * lane + 1) * dm.K + i] = civ.y;
              }
              __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
              __builtin_amdgcn_wave_barrier();
              __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
              ++nmerged;
              scan = true;
            }
            j0 = jj + 1;
          }
        }
      }
    }
    __syncthreads();
  }

  // recycling ranks: e-th empty slot in ascending order
  if (wave == 0) {
    if (lane == 0) s_cnt[1] = nmerged;
    // and the worklist of slots to recycle or refresh (in the pair list)
    int run = 0, nw = 0;
    for (int k0 = 0; k0 < A; k0 += 64) {
      const int k = k0 + lane;
      const bool empty = k < A && s_n[k] == 0;
      const bool work = k < A && (empty || s_dirty[k] != 0);
      const unsigned long long bal = __ballot(empty), bw = __ballot(work);
      if (empty) s_rk[k] = (uint16_t)(run + __popcll(bal & below));
      if (work) s_pairs[nw + __popcll(bw & below)] = (uint32_t)k;
      run += __popcll(bal);
      nw += __popcll(bw);
    }
    if (lane == 0) {
      s_cnt[2] = run;
      s_np = nw;
    }
  }
  __syncthreads();
  const int nwork = s_np;

  // 3. recycling and 4. screening copies
  const int ntok = dm.W * T;
  for (int x = wave; x < nwork; x += MT_WAVES) {  // uniform
    const int k = __builtin_amdgcn_readfirstlane((int)s_pairs[x]);
    uint8_t* row = rows + (size_t)k * ROW;
    if (s_n[k] == 0) {
      const int e = (int)s_rk[k] % ntok;
      const int f = t - e / T, j = e % T;
      const int rs = f % (dm.W + 1);
      const size_t tb = ((unit * (dm.W + 1) + rs) * (size_t)T + j) * D;
      const float2 kk = load2<FP32>(ws.ring_k, tb + 2 * lane);
      const float2 vv = load2<FP32>(ws.ring_v, tb + 2 * lane);
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
      m.tau = f * T + j;
      if (lane == 0) *reinterpret_cast<RowMeta*>(row + ROW_META) = m;
      refresh_cache(dm, kk, m, unit, k, ws, lane);
    } else if (s_dirty[k]) {
      const float2 sk = reinterpret_cast<const float2*>(row + ROW_SUMK)[lane];
      const RowMeta m = *reinterpret_cast<const RowMeta*>(row + ROW_META);
      refresh_cache(dm, sk, m, unit, k, ws, lane);
    }
  }
  if (tid == 0) {
    if (s_cnt[0]) atomicAdd(&ws.counters[CNT_AGED], (unsigned long long)s_cnt[0]);
    if (s_cnt[1]) atomicAdd(&ws.counters[CNT_MERGED], (unsigned long long)s_cnt[1]);
    if (s_cnt[2]) atomicAdd(&ws.counters[CNT_RECYCLED], (unsigned long long)s_cnt[2]);
  }
}

hipError_t launch_maintain(const Dims& dm, const Workspace& ws, const FoldBatch& fb, hipStream_t st) {
  const size_t lds = mt_lds_bytes(dm.K);  // <= 142 KiB for K <= MT_KMAX
  using KFn = void (*)(Dims, Workspace, FoldBatch);
  const int fd = mt_fd(dm.K);
  const KFn fn = dm.kv_fp32 ? (fd == 16 ? k_maintain<1, 16> : fd == 8 ? k_maintain<1, 8> : k_maintain<1, 4>)
                            : (fd == 16 ? k_maintain<0, 16> : fd == 8 ? k_maintain<0, 8> : k_maintain<0, 4>);
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(fn, dim3(fb.n * dm.units), dim3(MT_THREADS), lds, st, dm, ws, fb);
  return hipGetLastError();
}

}  // namespace pkv
