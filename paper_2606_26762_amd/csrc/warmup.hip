// PQ codebook warm-up (appendix "PQ codebook initialization"): during the
// first warm_frames folds of a stream the residuals of its assigned tokens
// are collected into a reservoir; after the last of them mini-batch k-means
// learns each (layer, kv head)'s key and value codebooks per subspace.
#include <hip/hip_runtime.h>

#include <cmath>

#include "pkv_internal.h"

namespace pkv {

// Residual collection, between the screen (which wrote the assignments) and
// the aggregation (which moves the centres): thread = (entry, unit, token j,
// K/V, 8 dims).  A non-seed token j of a warm-up fold goes to reservoir row
// rfill + (j - nseed) (while rows remain) as x - float32(sum / n) of its
// slot, the centre before this fold.
template <int FP32>
__global__ __launch_bounds__(256) void k_warm_collect(Dims dm, Workspace ws, FoldBatch fb) {
  const size_t gid = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t per = (size_t)dm.units * dm.T * 32;
  const int b = (int)(gid / per);
  if (b >= fb.n) return;
  const size_t r = gid % per;
  const int c = (int)(r & 15), side = (int)((r >> 4) & 1);
  const int j = (int)((r >> 5) % dm.T), u = (int)((r >> 5) / dm.T);
  if (!fb.warm[b] || j < fb.nseed[b]) return;
  const int row = fb.rfill[b] + (j - fb.nseed[b]);
  if (row >= dm.warm_tokens) return;
  const size_t unit = (size_t)fb.sid[b] * dm.units + u;
  const int slot = ws.assign[unit * dm.T + j];
  const uint8_t* brow = ws.bank + (unit * dm.K + slot) * ROW;
  const float nf = (float)reinterpret_cast<const RowMeta*>(brow + ROW_META)->n;
  const float* sum = reinterpret_cast<const float*>(brow + (side ? ROW_SUMV : ROW_SUMK)) + 8 * c;
  const size_t e = ((unit * (dm.W + 1) + fb.slot[b]) * dm.T + j) * (size_t)D + 8 * c;
  const uint8_t* ring = side ? ws.ring_v : ws.ring_k;
  float x[8];
  if (FP32) {
    const float4 a = reinterpret_cast<const float4*>(ring + e * 4)[0];
    const float4 q = reinterpret_cast<const float4*>(ring + e * 4)[1];
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = q.x; x[5] = q.y; x[6] = q.z; x[7] = q.w;
  } else {
    const uint4 w = *reinterpret_cast<const uint4*>(ring + e * 2);
    const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      x[2 * q] = __uint_as_float(ww[q] << 16);
      x[2 * q + 1] = __uint_as_float(ww[q] & 0xFFFF0000u);
    }
  }
  const float4 s0 = reinterpret_cast<const float4*>(sum)[0], s1 = reinterpret_cast<const float4*>(sum)[1];
  const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
  float res[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) res[q] = x[q] - sv[q] / nf;
  float* out = ws.reservoir + ((unit * 2 + side) * (size_t)dm.warm_tokens + row) * D + 8 * c;
  reinterpret_cast<float4*>(out)[0] = make_float4(res[0], res[1], res[2], res[3]);
  reinterpret_cast<float4*>(out)[1] = make_float4(res[4], res[5], res[6], res[7]);
}

// Mini-batch k-means, one wave per (entry, unit, K/V, subspace g) over the
// reservoir rows' 16 dims of g: centres start at rows i * floor(N / C); per
// batch of kmeans_batch consecutive rows each lane assigns one row to its
// nearest centre (float32 sequential distance over the dims, ties to the
// lower index) with the centres as the batch starts, then the rows update
// their centres in row order (count += 1, eta = 1 / count,
// c <- (1 - eta) c + eta x); kmeans_epochs passes.
// A row's count is known before any update: the count of its centre before
// the batch plus its rank among the batch's rows of that centre (ballots).
// So each row lane forms 1 - eta and eta x in parallel, and the row-order
// chain of a centre is one multiply and one add per row.  In that chain lane
// (kq, d) = (lane / 16, lane % 16) holds dim d of centres kq, kq + 4, kq + 8,
// kq + 12 in registers and takes each row's centre and 1 - eta from the row's
// lane (readlane); the next batch's rows are loaded during this one.
// The learned codewords replace the codebook, with its |C|^2 / 2 and the
// bound on max |C| that the PQ encoder uses.
__global__ __launch_bounds__(64) void k_warm_kmeans(Dims dm, Workspace ws, KmeansBatch kb) {
  __shared__ float s_c[CMAX][DP];
  __shared__ float s_ex[64][DP];  // eta x of each batch row
  __shared__ int s_cnt[CMAX];     // count of each centre before the batch
  const int lane = threadIdx.x;
  int id = blockIdx.x;
  const int g = id % G;
  id /= G;
  const int side = id & 1;
  id >>= 1;
  const int u = id % dm.units, e = id / dm.units;
  if (e >= kb.n) return;
  const int C = dm.C;
  const int N = min(kb.count[e], dm.warm_tokens);
  if (N < C) return;  // uniform: too few residuals, the given codebook stays
  const size_t unit = (size_t)kb.sid[e] * dm.units + u;
  const float* res = ws.reservoir + (unit * 2 + side) * (size_t)dm.warm_tokens * D + g * DP;
  for (int x = lane; x < CMAX * DP; x += 64)
    s_c[x / DP][x % DP] = x < C * DP ? res[(size_t)(x / DP) * (N / C) * D + x % DP] : 0.f;
  if (lane < CMAX) s_cnt[lane] = 0;
  const int d = lane & 15, kq = lane >> 4;
  float cr[CMAX / 4];  // dim d of centres kq + 4 m
  __syncthreads();
#pragma unroll
  for (int m = 0; m < CMAX / 4; ++m) cr[m] = s_c[kq + 4 * m][d];
  const unsigned long long below = (1ull << lane) - 1ull;
  const int B = dm.kmeans_batch;
  float xn[DP];  // this lane's row of the next batch
  auto load_row = [&](int b0) {
    if (lane < min(B, N - b0)) {
      const float4* src = reinterpret_cast<const float4*>(res + (size_t)(b0 + lane) * D);
#pragma unroll
      for (int q = 0; q < DP / 4; ++q) {
        const float4 v = src[q];
        xn[4 * q] = v.x; xn[4 * q + 1] = v.y; xn[4 * q + 2] = v.z; xn[4 * q + 3] = v.w;
      }
    }
  };
  load_row(0);
  for (int ep = 0; ep < dm.kmeans_epochs; ++ep) {
    for (int b0 = 0; b0 < N; b0 += B) {
      const int nb = min(B, N - b0);
      const bool row = lane < nb;
      float x[DP];
#pragma unroll
      for (int q = 0; q < DP; ++q) x[q] = xn[q];
      if (b0 + B < N) load_row(b0 + B);
      else if (ep + 1 < dm.kmeans_epochs) load_row(0);
      int bz = -1;
      if (row) {
        float best = INFINITY;
        bz = 0;
#pragma unroll
        for (int k = 0; k < CMAX; ++k) {
          if (k < C) {
            float acc = 0.f;
#pragma unroll
            for (int q = 0; q < DP; ++q) {
              const float df = x[q] - s_c[k][q];
              acc = acc + df * df;
            }
            if (acc < best) {
              best = acc;
              bz = k;
            }
          }
        }
      }
      // rank of this row among the batch's rows of its centre; lane k keeps
      // the number of rows of centre k
      int rank = 0, tot = 0;
      for (int k = 0; k < C; ++k) {
        const unsigned long long mk = __ballot(bz == k);
        if (bz == k) rank = __popcll(mk & below);
        if (lane == k) tot = __popcll(mk);
      }
      float om = 0.f;
      if (row) {
        const float eta = 1.0f / (float)(s_cnt[bz] + rank + 1);
        om = 1.0f - eta;
#pragma unroll
        for (int q = 0; q < DP; ++q) s_ex[lane][q] = eta * x[q];
      }
      __syncthreads();
      if (lane < C) s_cnt[lane] += tot;
      for (int i = 0; i < nb; ++i) {
        const int z = __builtin_amdgcn_readlane(bz, i);
        const float omi = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(om), i));
        const float ex = s_ex[i][d];
        const bool mine = (z & 3) == kq;
#pragma unroll
        for (int m = 0; m < CMAX / 4; ++m) {
          const float v = omi * cr[m] + ex;
          cr[m] = (mine && (z >> 2) == m) ? v : cr[m];
        }
      }
      // the assignments of the next batch read the updated centres
#pragma unroll
      for (int m = 0; m < CMAX / 4; ++m) s_c[kq + 4 * m][d] = cr[m];
      __syncthreads();
    }
  }
  float* cb = ws.codebooks + ((unit * 2 + side) * G + g) * (size_t)(CMAX * DP);
  for (int x = lane; x < C * DP; x += 64) cb[x] = s_c[x / DP][x % DP];
  // |C|^2 / 2 per codeword (float32 sequential fused multiply-add) and the
  // bound sqrt(max |C|^2) * 1.0001 of the subspace
  float n2 = 0.f;
  if (lane < C)
    for (int d = 0; d < DP; ++d) n2 = fmaf(s_c[lane][d], s_c[lane][d], n2);
  if (lane < CMAX) ws.cbhn[((unit * 2 + side) * G + g) * CMAX + lane] = lane < C ? 0.5f * n2 : 3e38f;
  float m = lane < C ? n2 : 0.f;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  if (lane == 0) ws.cbmax[(unit * 2 + side) * G + g] = sqrtf(m) * 1.0001f;
}

hipError_t launch_warm_collect(const Dims& dm, const Workspace& ws, const FoldBatch& fb, hipStream_t st) {
  const size_t n = (size_t)fb.n * dm.units * dm.T * 32;
  const dim3 grid((unsigned)((n + 255) / 256));
  if (dm.kv_fp32)
    hipLaunchKernelGGL(k_warm_collect<1>, grid, dim3(256), 0, st, dm, ws, fb);
  else
    hipLaunchKernelGGL(k_warm_collect<0>, grid, dim3(256), 0, st, dm, ws, fb);
  return hipGetLastError();
}

hipError_t launch_warm_kmeans(const Dims& dm, const Workspace& ws, const KmeansBatch& kb, hipStream_t st) {
  if (kb.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_warm_kmeans, dim3((unsigned)(kb.n * dm.units * 2 * G)), dim3(64), 0, st, dm, ws, kb);
  return hipGetLastError();
}

}  // namespace pkv
