// libprotokv host side: configuration checks, workspace carve-up, per-stream
// state machine and kernel sequencing on the caller's HIP stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "pkv_internal.h"

using namespace pkv;

namespace {

constexpr int MAX_ROWS = 512;  // query rows per kv head per attend call

struct StreamState {
  uint64_t frames = 0;
  uint64_t evicted = 0;
  int active = 0;
  bool pending = false;
  int pending_fe = -1;
  int folds = 0;  // folds done (the first warm_frames are the codebook warm-up)
  int rfill = 0;  // warm-up reservoir rows filled
};

struct Layout {
  size_t ring_k, ring_v, bank, chat_hi, chat_lo, cmeta, assign, codebooks, cbhn, cbmax;
  size_t pk, pv, pbias, pcodes, part_o, part_ml, counters, touched, ring_kr, qrot, rope_inv, reservoir, ema_res;
  size_t ps_count, ps_off, prow_bias, total;
};

thread_local std::string g_init_err;

size_t kv_bytes(const protokv_config& c) { return c.kv_dtype == PROTOKV_KV_FP32 ? 4 : 2; }

Layout make_layout(const protokv_config& c) {
  Layout ly{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += (bytes + 255) & ~(size_t)255;
    return o;
  };
  const size_t es = kv_bytes(c);
  const size_t units = (size_t)c.num_layers * c.num_kv_heads;
  const size_t U = (size_t)c.num_streams * units;
  const size_t T = (size_t)c.grid_h * c.grid_w;
  const size_t K = (size_t)c.capacity;
  const size_t S = (size_t)c.pseudo_per_proto;
  const size_t rows = (size_t)c.max_query_tokens * (c.num_q_heads / c.num_kv_heads);
  ly.ring_k = take(U * (c.window_frames + 1) * T * D * es);
  ly.ring_v = take(U * (c.window_frames + 1) * T * D * es);
  ly.bank = take(U * K * ROW);
  const size_t K32 = (size_t)cap32(c.capacity);
  ly.chat_hi = take(U * K32 * D * 2);
  ly.chat_lo = take(U * K32 * D * 2);
  ly.cmeta = take(U * K * CMETA_STRIDE * sizeof(CacheMeta));
  ly.assign = take(U * T * 4);
  ly.codebooks = take(U * 2 * G * CMAX * DP * 4);
  ly.cbhn = take(U * 2 * G * CMAX * 4);
  ly.cbmax = take(U * 2 * G * 4);
  ly.pk = take(units * K * S * D * es);
  ly.pv = take(units * K * S * D * es);
  ly.pbias = take(units * K * 4);
  ly.pcodes = take(units * K * 2 * PCW * 4);
  ly.part_o = take(units * MAX_SPLITS * rows * D * 4);
  ly.part_ml = take(units * MAX_SPLITS * rows * 2 * 4);
  ly.counters = take(CNT_COUNT * 8);
  ly.touched = take(U * K * 4);
  const bool rope = c.rope_theta > 0.0;
  ly.ring_kr = take(rope ? U * (c.window_frames + 1) * T * D * es : 0);
  ly.qrot = take(rope ? (size_t)c.num_layers * c.max_query_tokens * c.num_q_heads * D * es : 0);
  ly.rope_inv = take(rope ? (D / 2) * sizeof(double) : 0);
  ly.reservoir = take(c.warm_frames > 0 ? U * 2 * (size_t)c.warm_tokens * D * 4 : 0);
  ly.ema_res = take((c.flags & PROTOKV_FLAG_EMA_CENTRES) ? U * T * 2 * D * 4 : 0);
  const bool va = (c.flags & PROTOKV_FLAG_VAR_ALLOC) != 0;
  ly.ps_count = take(va ? units * K * 4 : 0);
  ly.ps_off = take(va ? units * K * 4 : 0);
  ly.prow_bias = take(va ? units * K * S * 4 : 0);
  ly.total = off;
  return ly;
}

// One stream's state blob (protokv.h): header, then 256-byte aligned sections.
struct StateLayout {
  size_t ring_k, ring_v, bank, codebooks, reservoir, ring_kr, total;
};

StateLayout state_layout(const protokv_config& c) {
  StateLayout sl{};
  size_t off = 256;  // the header, padded
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += (bytes + 255) & ~(size_t)255;
    return bytes ? o : (size_t)0;
  };
  const size_t units = (size_t)c.num_layers * c.num_kv_heads;
  const size_t T = (size_t)c.grid_h * c.grid_w;
  const size_t ring = units * (c.window_frames + 1) * T * D * kv_bytes(c);
  sl.ring_k = take(ring);
  sl.ring_v = take(ring);
  sl.bank = take(units * c.capacity * ROW);
  sl.codebooks = take(units * 2 * G * (size_t)c.pq_codewords * DP * 4);
  sl.reservoir = take(c.warm_frames > 0 ? units * 2 * (size_t)c.warm_tokens * D * 4 : 0);
  sl.ring_kr = take(c.rope_theta > 0.0 ? ring : 0);
  sl.total = off;
  return sl;
}

// Per codeword |C|^2 / 2 and per (K/V, subspace) a bound on max |C| of
// codebooks padded to CMAX codewords, for the PQ encoder's error bound
// (float32, sequential fused multiply-add).
void codebook_tables(const std::vector<float>& cb, int C, std::vector<float>& hn, std::vector<float>& cmax) {
  const size_t blocks = cb.size() / (CMAX * DP);
  hn.assign(blocks * CMAX, 0.f);
  cmax.assign(blocks, 0.f);
  for (size_t blk = 0; blk < blocks; ++blk) {
    float m = 0.f;
    for (int cc = 0; cc < CMAX; ++cc) {
      float n2 = 0.f;
      for (int q = 0; q < DP; ++q) n2 = std::fma(cb[(blk * CMAX + cc) * DP + q], cb[(blk * CMAX + cc) * DP + q], n2);
      hn[blk * CMAX + cc] = cc < C ? 0.5f * n2 : 3e38f;  // finite: the encoder tags scores
      if (cc < C) m = std::max(m, n2);
    }
    cmax[blk] = std::sqrt(m) * 1.0001f;
  }
}

// Codebooks [units][2][G][C][DP] -> the padded device layout [units][2][G][CMAX][DP].
std::vector<float> pad_codebooks(const float* codebooks, size_t units, int C) {
  std::vector<float> cb(units * 2 * G * CMAX * DP, 0.f);
  for (size_t uu = 0; uu < units; ++uu)
    for (int kv = 0; kv < 2; ++kv)
      for (int g = 0; g < G; ++g)
        for (int cc = 0; cc < C; ++cc)
          std::memcpy(&cb[(((uu * 2 + kv) * G + g) * CMAX + cc) * DP],
                      &codebooks[(((uu * 2 + kv) * G + g) * C + cc) * DP], DP * sizeof(float));
  return cb;
}

protokv_status check_config(const protokv_config* c, std::string& why) {
  if (!c) { why = "config is NULL"; return PROTOKV_E_INVALID; }
  auto bad = [&](const char* m) { why = m; return PROTOKV_E_INVALID; };
  auto uns = [&](const char* m) { why = m; return PROTOKV_E_UNSUPPORTED; };
  if (c->num_streams < 1) return bad("num_streams must be >= 1");
  if (c->num_layers < 1 || c->num_kv_heads < 1) return bad("num_layers and num_kv_heads must be >= 1");
  if (c->num_q_heads < c->num_kv_heads || c->num_q_heads % c->num_kv_heads)
    return bad("num_q_heads must be a positive multiple of num_kv_heads");
  if (c->head_dim != D) return uns("head_dim must be 128");
  if (c->grid_h < 1 || c->grid_w < 1) return bad("grid_h and grid_w must be >= 1");
  if ((int64_t)c->grid_h * c->grid_w > TMAX) return uns("at most 1024 tokens per frame");
  if (c->window_frames < 1) return bad("window_frames must be >= 1");
  if (c->capacity < 1) return bad("capacity must be >= 1");
  if (c->capacity > KMAX) return uns("capacity above 65535");
  if (c->pq_subspaces != G) return uns("pq_subspaces must be 8");
  if (c->pq_codewords < 2 || c->pq_codewords > CMAX) return uns("pq_codewords must be in [2, 16]");
  if (c->pseudo_per_proto < 1) return bad("pseudo_per_proto must be >= 1");
  if (c->pseudo_per_proto > SMAX) return uns("pseudo_per_proto above 16");
  if (c->beam < c->pseudo_per_proto) return bad("beam must be >= pseudo_per_proto");
  if (c->t_idle < 0) return bad("t_idle must be >= 0");
  if (c->max_query_tokens < 1) return bad("max_query_tokens must be >= 1");
  if ((int64_t)c->max_query_tokens * (c->num_q_heads / c->num_kv_heads) > MAX_ROWS)
    return uns("max_query_tokens * (num_q_heads/num_kv_heads) above 512");
  if (c->kv_dtype != PROTOKV_KV_BF16 && c->kv_dtype != PROTOKV_KV_FP32) return bad("kv_dtype unknown");
  if (c->flags & ~(uint32_t)(PROTOKV_FLAG_PQ | PROTOKV_FLAG_MASS_BIAS | PROTOKV_FLAG_MAINTENANCE |
                             PROTOKV_FLAG_EMA_CENTRES | PROTOKV_FLAG_MAH_SQUARED | PROTOKV_FLAG_VAR_ALLOC))
    return bad("unknown flag bits");
  if (c->flags & PROTOKV_FLAG_VAR_ALLOC) {
    if (c->pseudo_max < c->pseudo_per_proto) return bad("pseudo_max must be >= pseudo_per_proto");
    if (c->pseudo_max > SMAX) return uns("pseudo_max above 16");
    if (c->beam < c->pseudo_max) return bad("beam must be >= pseudo_max");
    if (c->capacity > AL_KMAX) return uns("the variance-aware allocation supports capacity up to 4096");
  }
  if (c->flags & PROTOKV_FLAG_EMA_CENTRES) {
    if (!(c->alpha >= 0.f && c->alpha <= 1.f) || !(c->beta >= 0.f && c->beta <= 1.f))
      return bad("alpha and beta must be in [0, 1]");
    if (c->flags & PROTOKV_FLAG_MAINTENANCE) return uns("maintenance with EMA centres");
  }
  if (!(c->rope_theta == 0.0 || (c->rope_theta > 1.0 && std::isfinite(c->rope_theta))))
    return bad("rope_theta must be 0 (off) or a finite base > 1");
  if (c->warm_frames < 0) return bad("warm_frames must be >= 0");
  if (c->warm_frames > 0) {
    if (c->warm_tokens < 1 || c->warm_tokens > 65536) return bad("warm_tokens must be in [1, 65536]");
    if (c->kmeans_epochs < 1) return bad("kmeans_epochs must be >= 1");
    if (c->kmeans_batch < 1 || c->kmeans_batch > 64) return bad("kmeans_batch must be in [1, 64]");
    if (!(c->flags & PROTOKV_FLAG_PQ)) return bad("the codebook warm-up needs PROTOKV_FLAG_PQ");
    if (c->flags & PROTOKV_FLAG_EMA_CENTRES) return uns("codebook warm-up with EMA centres");
  }
  if (!(c->eta > 0.f && c->eta < 1.f)) return bad("eta must be in (0, 1)");
  if (c->pq_eps != 1.0f) return uns("pq_eps must be 1");
  if (!(c->lambda_sp >= 0.0) || !(c->lambda_idle >= 0.0) || !std::isfinite(c->lambda_sp) ||
      !std::isfinite(c->lambda_idle))
    return bad("lambda_sp and lambda_idle must be finite and >= 0");
  if (!(c->ridge > 0.0) || !std::isfinite(c->ridge)) return bad("ridge must be finite and > 0");
  if (c->flags & PROTOKV_FLAG_MAINTENANCE) {
    if (!(c->gamma >= 0.0 && c->gamma < 1.0)) return bad("gamma must be in [0, 1)");
    if (!(c->eps_k >= 0.0) || !(c->eps_v >= 0.0) || !std::isfinite(c->eps_k) || !std::isfinite(c->eps_v))
      return bad("eps_k and eps_v must be finite and >= 0");
    if (c->capacity > MT_KMAX) return uns("maintenance supports capacity up to 2048");
  }
  return PROTOKV_OK;
}

}  // namespace

struct protokv_ctx {
  protokv_config cfg;
  Dims dm;
  Workspace ws;
  Layout ly;
  uint8_t* base = nullptr;
  std::vector<StreamState> st;
  void* scratch = nullptr;  // this device's protokv_attend_static array
  int synth_stream = -1;
  int synth_active = 0;
  bool synth_rows = false;  // pseudo-token rows written (else only centres, biases, codes)
  uint64_t folds = 0, assigned = 0, seeded = 0;
  std::string err;
  // per-kernel event timing (diagnostics)
  uint32_t profile_mask = 0;
  std::vector<hipEvent_t> ev_pool;
  struct Timed { int id; hipEvent_t a, b; };
  std::vector<Timed> timed;
  size_t ev_next = 0;

  template <class F>
  hipError_t launch(int id, hipStream_t st, F&& f) {
    if (!(profile_mask >> id & 1u)) return f();
    hipEvent_t e[2];
    for (int i = 0; i < 2; ++i) {
      if (ev_next == ev_pool.size()) {
        hipEvent_t ne;
        hipError_t r = hipEventCreateWithFlags(&ne, hipEventDisableSystemFence);
        if (r != hipSuccess) return r;
        ev_pool.push_back(ne);
      }
      e[i] = ev_pool[ev_next++];
    }
    hipError_t r = hipEventRecord(e[0], st);
    if (r == hipSuccess) r = f();
    if (r == hipSuccess) r = hipEventRecord(e[1], st);
    if (r == hipSuccess) timed.push_back({id, e[0], e[1]});
    return r;
  }
  ~protokv_ctx() {
    for (hipEvent_t e : ev_pool) (void)hipEventDestroy(e);
  }

  protokv_status fail(protokv_status s, const std::string& m) {
    err = m;
    return s;
  }
  protokv_status dev(hipError_t e, const char* where) {
    if (e == hipSuccess) return PROTOKV_OK;
    err = std::string(where) + ": " + hipGetErrorString(e);
    return PROTOKV_E_DEVICE;
  }
};

extern "C" {

protokv_status protokv_default_config(protokv_config* c) {
  if (!c) return PROTOKV_E_INVALID;
  std::memset(c, 0, sizeof(*c));
  c->num_streams = 1;
  c->num_layers = 28;
  c->num_kv_heads = 4;
  c->num_q_heads = 28;
  c->head_dim = 128;
  c->grid_h = 14;
  c->grid_w = 14;
  c->window_frames = 8;
  c->capacity = 256;
  c->pseudo_per_proto = 8;
  c->pq_subspaces = 8;
  c->pq_codewords = 16;
  c->beam = 32;
  c->t_idle = 120;
  c->max_query_tokens = 64;
  c->kv_dtype = PROTOKV_KV_BF16;
  c->flags = PROTOKV_FLAG_PQ | PROTOKV_FLAG_MASS_BIAS;
  c->eta = 0.05f;
  c->pq_eps = 1.0f;
  c->lambda_sp = 0.1;
  c->lambda_idle = 0.01;
  c->ridge = 1e-4;
  c->gamma = 0.05;
  c->eps_k = 0.20;
  c->eps_v = 0.25;
  c->alpha = 0.05f;
  c->beta = 0.05f;
  c->warm_tokens = 1024;
  c->kmeans_epochs = 4;
  c->kmeans_batch = 64;
  c->pseudo_max = 16;
  return PROTOKV_OK;
}

protokv_status protokv_validate_config(const protokv_config* c) {
  std::string why;
  protokv_status s = check_config(c, why);
  if (s != PROTOKV_OK) g_init_err = why;
  return s;
}

protokv_status protokv_workspace_size(const protokv_config* c, size_t* bytes) {
  std::string why;
  protokv_status s = check_config(c, why);
  if (s != PROTOKV_OK) { g_init_err = why; return s; }
  if (!bytes) { g_init_err = "bytes is NULL"; return PROTOKV_E_INVALID; }
  *bytes = make_layout(*c).total;
  return PROTOKV_OK;
}

protokv_status protokv_init(const protokv_config* c, const float* codebooks, void* workspace,
                            size_t workspace_bytes, void* stream, protokv_t* out) {
  std::string why;
  protokv_status s = check_config(c, why);
  if (s != PROTOKV_OK) { g_init_err = why; return s; }
  if (!out) { g_init_err = "out is NULL"; return PROTOKV_E_INVALID; }
  if (!codebooks) { g_init_err = "codebooks is NULL"; return PROTOKV_E_INVALID; }
  Layout ly = make_layout(*c);
  if (!workspace) { g_init_err = "workspace is NULL"; return PROTOKV_E_WORKSPACE; }
  if ((uintptr_t)workspace % 256) { g_init_err = "workspace must be 256-byte aligned"; return PROTOKV_E_WORKSPACE; }
  if (workspace_bytes < ly.total) {
    g_init_err = "workspace too small: need " + std::to_string(ly.total) + " bytes";
    return PROTOKV_E_WORKSPACE;
  }
  hipStream_t hs = (hipStream_t)stream;
  auto* h = new protokv_ctx();
  h->cfg = *c;
  h->ly = ly;
  h->base = (uint8_t*)workspace;
  Dims& dm = h->dm;
  dm.L = c->num_layers;
  dm.Hkv = c->num_kv_heads;
  dm.Hq = c->num_q_heads;
  dm.T = c->grid_h * c->grid_w;
  dm.grid_h = c->grid_h;
  dm.grid_w = c->grid_w;
  dm.W = c->window_frames;
  dm.K = c->capacity;
  dm.S = c->pseudo_per_proto;
  dm.C = c->pq_codewords;
  dm.t_idle = c->t_idle;
  dm.units = c->num_layers * c->num_kv_heads;
  dm.streams = c->num_streams;
  dm.kv_fp32 = c->kv_dtype == PROTOKV_KV_FP32;
  dm.flags = c->flags;
  dm.eta = c->eta;
  dm.lambda_sp = c->lambda_sp;
  dm.lambda_idle = c->lambda_idle;
  dm.ridge = c->ridge;
  dm.gamma = c->gamma;
  dm.eps_k = c->eps_k;
  dm.eps_v = c->eps_v;
  dm.alpha = c->alpha;
  dm.beta = c->beta;
  dm.rope_theta = c->rope_theta;
  dm.warm_frames = c->warm_frames;
  dm.warm_tokens = c->warm_tokens;
  dm.kmeans_epochs = c->kmeans_epochs;
  dm.kmeans_batch = c->kmeans_batch;
  dm.pseudo_max = c->pseudo_max;
  dm.max_rows = c->max_query_tokens * (c->num_q_heads / c->num_kv_heads);
  dm.max_splits = MAX_SPLITS;
  uint8_t* b = h->base;
  Workspace& ws = h->ws;
  ws.ring_k = b + ly.ring_k;
  ws.ring_v = b + ly.ring_v;
  ws.bank = b + ly.bank;
  ws.chat_hi = (uint16_t*)(b + ly.chat_hi);
  ws.chat_lo = (uint16_t*)(b + ly.chat_lo);
  ws.cmeta = (CacheMeta*)(b + ly.cmeta);
  ws.assign = (int32_t*)(b + ly.assign);
  ws.codebooks = (float*)(b + ly.codebooks);
  ws.cbhn = (float*)(b + ly.cbhn);
  ws.cbmax = (float*)(b + ly.cbmax);
  ws.pk = b + ly.pk;
  ws.pv = b + ly.pv;
  ws.pbias = (float*)(b + ly.pbias);
  ws.pcodes = (uint32_t*)(b + ly.pcodes);
  ws.part_o = (float*)(b + ly.part_o);
  ws.part_ml = (float*)(b + ly.part_ml);
  ws.counters = (unsigned long long*)(b + ly.counters);
  ws.touched = (uint32_t*)(b + ly.touched);
  const bool rope = c->rope_theta > 0.0;
  ws.ring_kr = rope ? b + ly.ring_kr : nullptr;
  ws.qrot = rope ? b + ly.qrot : nullptr;
  ws.rope_inv = rope ? (const double*)(b + ly.rope_inv) : nullptr;
  ws.reservoir = c->warm_frames > 0 ? (float*)(b + ly.reservoir) : nullptr;
  ws.ema_res = (c->flags & PROTOKV_FLAG_EMA_CENTRES) ? (float*)(b + ly.ema_res) : nullptr;
  const bool va = (c->flags & PROTOKV_FLAG_VAR_ALLOC) != 0;
  ws.ps_count = va ? (int32_t*)(b + ly.ps_count) : nullptr;
  ws.ps_off = va ? (int32_t*)(b + ly.ps_off) : nullptr;
  ws.prow_bias = va ? (float*)(b + ly.prow_bias) : nullptr;
  h->st.assign(c->num_streams, StreamState());

  // codebooks -> [U][2][G][CMAX][DP] with the codeword axis padded to 16
  const size_t U = (size_t)c->num_streams * dm.units;
  std::vector<float> cb = pad_codebooks(codebooks, U, c->pq_codewords), hn, cmax;
  codebook_tables(cb, c->pq_codewords, hn, cmax);
  hipError_t e = hipMemsetAsync(workspace, 0, ly.total, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(ws.codebooks, cb.data(), cb.size() * sizeof(float),
                                          hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(ws.cbhn, hn.data(), hn.size() * sizeof(float),
                                          hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(ws.cbmax, cmax.data(), cmax.size() * sizeof(float),
                                          hipMemcpyHostToDevice, hs);
  // rotary frequencies theta^(-2i/D) in float64
  std::vector<double> inv(D / 2);
  for (int i = 0; i < D / 2; ++i) inv[i] = std::pow(c->rope_theta, -2.0 * i / D);
  if (e == hipSuccess && ws.rope_inv)
    e = hipMemcpyAsync(const_cast<double*>(ws.rope_inv), inv.data(), inv.size() * sizeof(double),
                       hipMemcpyHostToDevice, hs);
  // the address of this device's protokv_attend_static scratch (once per device)
  if (e == hipSuccess) e = static_scratch_ptr(&h->scratch);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) {
    g_init_err = std::string("init: ") + hipGetErrorString(e);
    delete h;
    return PROTOKV_E_DEVICE;
  }
  *out = h;
  return PROTOKV_OK;
}

protokv_status protokv_destroy(protokv_t h) {
  if (!h) return PROTOKV_E_INVALID;
  delete h;
  return PROTOKV_OK;
}

protokv_status protokv_append_frame(protokv_t h, const int32_t* ids, int32_t n, const void* k,
                                    const void* v, void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  if (n < 1 || !ids || !k || !v) return h->fail(PROTOKV_E_INVALID, "append: need n >= 1 and non-NULL ids, k, v");
  std::vector<char> seen(h->cfg.num_streams, 0);
  for (int i = 0; i < n; ++i) {
    const int s = ids[i];
    if (s < 0 || s >= h->cfg.num_streams) return h->fail(PROTOKV_E_INVALID, "append: stream id out of range");
    if (seen[s]) return h->fail(PROTOKV_E_INVALID, "append: stream listed twice");
    seen[s] = 1;
    if (h->st[s].pending) return h->fail(PROTOKV_E_STATE, "append: stream has an unfolded eviction; call protokv_fold");
    if ((h->st[s].frames + 2) * (uint64_t)h->dm.T >= (1ull << 31))
      return h->fail(PROTOKV_E_UNSUPPORTED, "append: stream position exceeds 2^31 tokens");
    if (h->st[s].frames + 1 > (uint64_t)h->dm.W &&
        h->st[s].evicted + (uint64_t)h->dm.T > PROTOKV_MAX_EVICTED_TOKENS)
      return h->fail(PROTOKV_E_UNSUPPORTED,
                     "append: the stream would evict more than PROTOKV_MAX_EVICTED_TOKENS tokens per unit "
                     "(the exact decode's 192-bit products)");
  }
  hipStream_t hs = (hipStream_t)stream;
  const size_t entry_bytes = (size_t)h->dm.units * h->dm.T * D * kv_bytes(h->cfg);
  for (int b0 = 0; b0 < n; b0 += MAXB) {
    AppendBatch ab{};
    ab.n = std::min(MAXB, n - b0);
    for (int i = 0; i < ab.n; ++i) {
      const StreamState& ss = h->st[ids[b0 + i]];
      ab.sid[i] = ids[b0 + i];
      ab.slot[i] = (int)(ss.frames % (uint64_t)(h->dm.W + 1));
      ab.frame[i] = (int)ss.frames;
    }
    const uint8_t* kb = (const uint8_t*)k + b0 * entry_bytes;
    const uint8_t* vb = (const uint8_t*)v + b0 * entry_bytes;
    // with rotary positions the rotated copy of the keys is written in the same pass
    protokv_status s = h->dev(
        h->ws.ring_kr
            ? h->launch(PROTOKV_K_ROPE_RING, hs, [&] { return launch_ring_insert_rope(h->dm, h->ws, ab, kb, vb, hs); })
            : h->launch(PROTOKV_K_RING_INSERT, hs, [&] { return launch_ring_insert(h->dm, h->ws, ab, kb, vb, hs); }),
        "append");
    if (s != PROTOKV_OK) return s;
  }
  for (int i = 0; i < n; ++i) {
    StreamState& ss = h->st[ids[i]];
    ss.frames += 1;
    if (ss.frames > (uint64_t)h->dm.W) {
      ss.pending = true;
      ss.pending_fe = (int)(ss.frames - 1 - h->dm.W);
    }
  }
  return PROTOKV_OK;
}

protokv_status protokv_fold(protokv_t h, void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  hipStream_t hs = (hipStream_t)stream;
  std::vector<int> pend;
  for (int s = 0; s < h->cfg.num_streams; ++s)
    if (h->st[s].pending) pend.push_back(s);
  if (pend.empty()) return PROTOKV_OK;
  const int T = h->dm.T, K = h->dm.K;
  for (size_t b0 = 0; b0 < pend.size(); b0 += MAXB) {
    FoldBatch fb{};
    fb.n = (int)std::min<size_t>(MAXB, pend.size() - b0);
    int max_seed = 0;
    bool any_assign = false, any_warm = false;
    for (int i = 0; i < fb.n; ++i) {
      const int s = pend[b0 + i];
      const StreamState& ss = h->st[s];
      fb.sid[i] = s;
      fb.fe[i] = ss.pending_fe;
      fb.slot[i] = ss.pending_fe % (h->dm.W + 1);
      fb.t[i] = (int)(ss.frames - 1);
      fb.nact[i] = ss.active;
      fb.nseed[i] = std::min(T, K - ss.active);
      fb.warm[i] = ss.folds < h->dm.warm_frames ? 1 : 0;
      fb.rfill[i] = ss.rfill;
      max_seed = std::max(max_seed, fb.nseed[i]);
      any_assign |= fb.nseed[i] < T;
      any_warm |= fb.warm[i] && fb.nseed[i] < T;
    }
    protokv_status st = PROTOKV_OK;
    if (max_seed > 0)
      st = h->dev(h->launch(PROTOKV_K_SEED, hs, [&] { return launch_seed(h->dm, h->ws, fb, max_seed, hs); }),
                  "fold/seed");
    if (st == PROTOKV_OK && any_assign)
      st = h->dev(h->launch(PROTOKV_K_SCREEN, hs, [&] { return launch_screen(h->dm, h->ws, fb, hs); }),
                  "fold/screen");
    // warm-up folds: residuals against the centres before this fold
    if (st == PROTOKV_OK && any_warm)
      st = h->dev(h->launch(PROTOKV_K_WARM_COLLECT, hs, [&] { return launch_warm_collect(h->dm, h->ws, fb, hs); }),
                  "fold/warm-up collect");
    if (st == PROTOKV_OK && any_assign)
      st = h->dev(h->launch(PROTOKV_K_AGGREGATE, hs, [&] { return launch_aggregate(h->dm, h->ws, fb, hs); }),
                  "fold/aggregate");
    if (st == PROTOKV_OK && (h->dm.flags & PROTOKV_FLAG_MAINTENANCE))
      st = h->dev(h->launch(PROTOKV_K_MAINTAIN, hs, [&] { return launch_maintain(h->dm, h->ws, fb, hs); }),
                  "fold/maintain");
    // streams whose warm-up ends with this fold learn their codebooks
    KmeansBatch kb{};
    for (int i = 0; i < fb.n; ++i) {
      if (!fb.warm[i]) continue;
      const StreamState& ss = h->st[fb.sid[i]];
      if (ss.folds + 1 == h->dm.warm_frames) {
        kb.sid[kb.n] = fb.sid[i];
        kb.count[kb.n] = std::min(h->dm.warm_tokens, ss.rfill + (T - fb.nseed[i]));
        ++kb.n;
      }
    }
    if (st == PROTOKV_OK && kb.n > 0)
      st = h->dev(h->launch(PROTOKV_K_WARM_KMEANS, hs, [&] { return launch_warm_kmeans(h->dm, h->ws, kb, hs); }),
                  "fold/warm-up k-means");
    if (st != PROTOKV_OK) return st;
    for (int i = 0; i < fb.n; ++i) {
      StreamState& ss = h->st[fb.sid[i]];
      if (fb.warm[i]) ss.rfill = std::min(h->dm.warm_tokens, ss.rfill + (T - fb.nseed[i]));
      ss.folds += 1;
      ss.active += fb.nseed[i];
      ss.evicted += T;
      ss.pending = false;
      h->seeded += (uint64_t)fb.nseed[i] * h->dm.units;
      h->assigned += (uint64_t)(T - fb.nseed[i]) * h->dm.units;
      if (h->synth_stream == fb.sid[i]) h->synth_stream = -1;
    }
  }
  h->folds += 1;
  return PROTOKV_OK;
}

protokv_status protokv_synthesize(protokv_t h, int32_t sid, void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  if (sid < 0 || sid >= h->cfg.num_streams) return h->fail(PROTOKV_E_INVALID, "synthesize: stream id out of range");
  if (h->st[sid].pending) return h->fail(PROTOKV_E_STATE, "synthesize: stream has an unfolded eviction");
  hipStream_t hs = (hipStream_t)stream;
  const int na = h->st[sid].active;
  const bool va = h->ws.ps_count != nullptr;
  // bf16 with S >= PS_MIN_S: the decode also writes the float32 centres and
  // the readout forms the rows from them as it loads them; otherwise the rows
  // are written here
  // (with rotary positions the readout turns the formed pseudo-keys at tau_k;
  // with the variance-aware allocation each slot's S_k rows are written)
  const bool rows = h->dm.kv_fp32 != 0 || h->dm.S < PS_MIN_S || va;
  // a slot's residual count is at most the tokens its stream has evicted
  const bool wide = h->st[sid].evicted > 65534u;
  // the allocation decodes every slot's top pseudo_max tuples; slot k keeps its first S_k
  Dims dd = h->dm;
  if (va) dd.S = h->dm.pseudo_max;
  protokv_status s = h->dev(
      h->launch(PROTOKV_K_SYNTHESIZE, hs, [&] { return launch_decode(dd, h->ws, sid, na, !rows, wide, hs); }),
      "synthesize/decode");
  if (s == PROTOKV_OK && va)
    s = h->dev(h->launch(PROTOKV_K_ALLOC, hs, [&] { return launch_alloc(h->dm, h->ws, sid, na, hs); }),
               "synthesize/allocate");
  if (s == PROTOKV_OK && rows)
    s = h->dev(h->launch(PROTOKV_K_MATERIALIZE, hs, [&] { return launch_materialize(h->dm, h->ws, sid, na, hs); }),
               "synthesize/materialize");
  if (s != PROTOKV_OK) return s;
  h->synth_stream = sid;
  h->synth_active = h->st[sid].active;
  h->synth_rows = rows;
  return PROTOKV_OK;
}

// Checks a readout of stream sid and plans its context splits (at most
// max_splits); no launches.
static protokv_status plan_attend(protokv_t h, int32_t sid, const void* q, int32_t tq, void* o, float* lse,
                                  int max_splits, AttendArgs& aa, const char* who) {
  if (sid < 0 || sid >= h->cfg.num_streams) return h->fail(PROTOKV_E_INVALID, std::string(who) + ": stream id out of range");
  if (!q || !o) return h->fail(PROTOKV_E_INVALID, std::string(who) + ": q and o must be non-NULL");
  if (tq < 1 || tq > h->cfg.max_query_tokens)
    return h->fail(PROTOKV_E_INVALID, std::string(who) + ": tq outside [1, max_query_tokens]");
  const StreamState& ss = h->st[sid];
  if (ss.pending) return h->fail(PROTOKV_E_STATE, std::string(who) + ": stream has an unfolded eviction");
  if (h->synth_stream != sid)
    return h->fail(PROTOKV_E_STATE, std::string(who) + ": no synthesis of this stream since its last fold");
  aa = AttendArgs{};
  aa.sid = sid;
  const int T = h->dm.T, W = h->dm.W;
  const uint64_t nf = std::min<uint64_t>(ss.frames, (uint64_t)W);
  aa.f_first = (int)(ss.frames - nf);
  aa.n_near = (int)nf * T;
  aa.n_far = h->synth_active * h->dm.S;
  aa.gen = h->synth_rows ? 0 : 1;
  aa.tq = tq;
  aa.q = q;
  aa.near_k = h->ws.ring_kr ? h->ws.ring_kr : h->ws.ring_k;
  aa.rowbias = h->ws.prow_bias;
  aa.o = o;
  aa.lse = lse;
  const int ctx = aa.n_near + aa.n_far;
  if (ctx == 0) return h->fail(PROTOKV_E_STATE, std::string(who) + ": empty context (no frames appended)");
  const int rows = tq * (h->dm.Hq / h->dm.Hkv);
  int splits;
  if (h->dm.kv_fp32) splits = std::max(1, std::min(max_splits, (1024 + h->dm.units * rows - 1) / (h->dm.units * rows)));
  else {
    const int rblocks = (rows + 255) / 256;
    // about one workgroup per compute unit (256 on MI355X)
    splits = std::max(1, std::min(max_splits, (256 + h->dm.units * rblocks / 2) / (h->dm.units * rblocks)));
  }
  auto up64 = [](int x) { return (x + 63) / 64 * 64; };
  if (aa.gen) {
    // pseudo-token rows formed in LDS (bf16): every split takes an equal
    // share of the near-window tiles and of the formed tiles, which cost
    // more than the tiles loaded directly
    aa.near_chunk = std::max(64, up64((aa.n_near + splits - 1) / splits));
    aa.far_chunk = std::max(64, up64((aa.n_far + splits - 1) / splits));
    aa.splits = std::max((aa.n_near + aa.near_chunk - 1) / aa.near_chunk,
                         (aa.n_far + aa.far_chunk - 1) / aa.far_chunk);
    aa.chunk = 0;
    return PROTOKV_OK;
  }
  const int chunk = up64((ctx + splits - 1) / splits);
  aa.splits = (ctx + chunk - 1) / chunk;
  aa.chunk = chunk;
  return PROTOKV_OK;
}

// Enqueues a planned readout: the rotated query (rotary positions), the
// split readout and the merge, with the scratch of `ws` and the partial
// strides of `dm`.
static protokv_status run_attend(protokv_t h, const Dims& dm, const Workspace& ws, AttendArgs& aa, hipStream_t hs) {
  if (ws.qrot) {
    // rotary positions: the query rotated at P + t with P = frames appended * T
    const void* q = aa.q;
    const long long p0 = (long long)h->st[aa.sid].frames * dm.T;
    protokv_status sr = h->dev(
        h->launch(PROTOKV_K_ROPE_Q, hs, [&] { return launch_rope_q(dm, ws, q, aa.tq, p0, hs); }), "attend/rope");
    if (sr != PROTOKV_OK) return sr;
    aa.q = ws.qrot;
  }
  protokv_status s = h->dev(h->launch(PROTOKV_K_ATTEND, hs, [&] { return launch_attend(dm, ws, aa, hs); }),
                            "attend");
  if (s != PROTOKV_OK) return s;
  return h->dev(h->launch(PROTOKV_K_ATTEND_MERGE, hs, [&] { return launch_attend_merge(dm, ws, aa, hs); }),
                "attend/merge");
}

protokv_status protokv_attend(protokv_t h, int32_t sid, const void* q, int32_t tq, void* o, float* lse,
                              void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  AttendArgs aa;
  protokv_status s = plan_attend(h, sid, q, tq, o, lse, MAX_SPLITS, aa, "attend");
  if (s != PROTOKV_OK) return s;
  return run_attend(h, h->dm, h->ws, aa, (hipStream_t)stream);
}

protokv_status protokv_attend_static(protokv_t h, int32_t sid, const void* q, int32_t tq, void* o, float* lse,
                                     void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  if (!h->scratch) return h->fail(PROTOKV_E_DEVICE, "attend_static: no scratch address for this device");
  const int rows = tq * (h->dm.Hq / h->dm.Hkv);
  const size_t es = kv_bytes(h->cfg);
  const size_t qrot = h->ws.qrot ? ((size_t)h->dm.L * std::max(tq, 1) * h->dm.Hq * D * es + 255) / 256 * 256 : 0;
  // partial outputs [units][splits][rows][D] and (m, l) [units][splits][rows][2], float32
  auto part_bytes = [&](int sp) {
    const size_t po = ((size_t)h->dm.units * sp * std::max(rows, 1) * D * 4 + 255) / 256 * 256;
    const size_t pm = ((size_t)h->dm.units * sp * std::max(rows, 1) * 2 * 4 + 255) / 256 * 256;
    return po + pm;
  };
  int max_splits = MAX_SPLITS;
  while (max_splits > 1 && part_bytes(max_splits) + qrot > PROTOKV_STATIC_SCRATCH_BYTES) --max_splits;
  if (part_bytes(1) + qrot > PROTOKV_STATIC_SCRATCH_BYTES)
    return h->fail(PROTOKV_E_UNSUPPORTED, "attend_static: the partials of one context split (units * rows * (D + 2) "
                                          "* 4 bytes) and the rotated query exceed PROTOKV_STATIC_SCRATCH_BYTES");
  AttendArgs aa;
  protokv_status s = plan_attend(h, sid, q, tq, o, lse, max_splits, aa, "attend_static");
  if (s != PROTOKV_OK) return s;
  // the same kernels with compact partial strides and the scratch pointers
  Dims dm = h->dm;
  dm.max_splits = aa.splits;
  dm.max_rows = rows;
  Workspace ws = h->ws;
  uint8_t* base = (uint8_t*)h->scratch;
  ws.part_o = (float*)base;
  ws.part_ml = (float*)(base + ((size_t)dm.units * aa.splits * rows * D * 4 + 255) / 256 * 256);
  if (ws.qrot) ws.qrot = base + part_bytes(aa.splits);
  return run_attend(h, dm, ws, aa, (hipStream_t)stream);
}

protokv_status protokv_stream_info_get(protokv_t h, int32_t sid, protokv_stream_info* out) {
  if (!h || !out) return PROTOKV_E_INVALID;
  if (sid < 0 || sid >= h->cfg.num_streams) return h->fail(PROTOKV_E_INVALID, "stream id out of range");
  const StreamState& ss = h->st[sid];
  out->frames = ss.frames;
  out->evicted_tokens = ss.evicted;
  out->active_slots = ss.active;
  out->pending = ss.pending ? 1 : 0;
  return PROTOKV_OK;
}

protokv_status protokv_get_counters(protokv_t h, protokv_counters* out, void* stream) {
  if (!h || !out) return PROTOKV_E_INVALID;
  unsigned long long dc[CNT_COUNT];
  hipStream_t hs = (hipStream_t)stream;
  hipError_t e = hipMemcpyAsync(dc, h->ws.counters, sizeof(dc), hipMemcpyDeviceToHost, hs);
  const size_t nt = (size_t)h->cfg.num_streams * h->dm.units * h->dm.K;
  std::vector<uint32_t> tv(nt);
  if (e == hipSuccess) e = hipMemcpyAsync(tv.data(), h->ws.touched, nt * 4, hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return h->dev(e, "get_counters");
  uint64_t touched = 0;
  for (uint32_t x : tv) touched += x;
  out->folds = h->folds;
  out->tokens_assigned = h->assigned;
  out->tokens_seeded = h->seeded;
  out->refined = dc[CNT_REFINED];
  out->refined_full = dc[CNT_REFINED_FULL];
  out->near_ties = dc[CNT_NEAR_TIES];
  out->touched = touched;
  out->aged = dc[CNT_AGED];
  out->merged = dc[CNT_MERGED];
  out->recycled = dc[CNT_RECYCLED];
  return PROTOKV_OK;
}

static protokv_status copy_out(protokv_t h, void* dst, const void* src, size_t bytes, void* stream,
                               const char* where) {
  hipStream_t hs = (hipStream_t)stream;
  hipError_t e = hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  return h->dev(e, where);
}

protokv_status protokv_read_assignments(protokv_t h, int32_t sid, int32_t* dst, size_t count, void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  if (sid < 0 || sid >= h->cfg.num_streams || !dst) return h->fail(PROTOKV_E_INVALID, "read_assignments: bad stream or dst");
  const size_t n = (size_t)h->dm.units * h->dm.T;
  if (count != n) return h->fail(PROTOKV_E_INVALID, "read_assignments: count must be num_layers*num_kv_heads*T");
  return copy_out(h, dst, h->ws.assign + (size_t)sid * n, n * 4, stream, "read_assignments");
}

protokv_status protokv_read_codebooks(protokv_t h, int32_t sid, float* dst, size_t count, void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  if (sid < 0 || sid >= h->cfg.num_streams || !dst) return h->fail(PROTOKV_E_INVALID, "read_codebooks: bad stream or dst");
  const int C = h->dm.C;
  const size_t blocks = (size_t)h->dm.units * 2 * G;
  if (count != blocks * C * DP) return h->fail(PROTOKV_E_INVALID, "read_codebooks: count must be L*Hkv*2*G*C*(D/G)");
  std::vector<float> raw(blocks * CMAX * DP);
  protokv_status s = copy_out(h, raw.data(), h->ws.codebooks + (size_t)sid * blocks * CMAX * DP,
                              raw.size() * sizeof(float), stream, "read_codebooks");
  if (s != PROTOKV_OK) return s;
  for (size_t blk = 0; blk < blocks; ++blk)
    std::memcpy(dst + blk * C * DP, raw.data() + blk * CMAX * DP, (size_t)C * DP * sizeof(float));
  return PROTOKV_OK;
}

protokv_status protokv_read_bank(protokv_t h, int32_t sid, void* dst, size_t bytes, void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  if (sid < 0 || sid >= h->cfg.num_streams || !dst) return h->fail(PROTOKV_E_INVALID, "read_bank: bad stream or dst");
  const size_t n = (size_t)h->dm.units * h->dm.K * ROW;
  if (bytes != n) return h->fail(PROTOKV_E_INVALID, "read_bank: bytes must be units*capacity*PROTOKV_ROW_BYTES");
  return copy_out(h, dst, h->ws.bank + (size_t)sid * n, n, stream, "read_bank");
}

protokv_status protokv_read_pseudo(protokv_t h, void* keys, void* values, float* bias, void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  if (h->synth_stream < 0) return h->fail(PROTOKV_E_STATE, "read_pseudo: no synthesis since the last fold");
  const size_t n = (size_t)h->dm.units * h->dm.K * h->dm.S * D * kv_bytes(h->cfg);
  protokv_status s = PROTOKV_OK;
  if (!h->synth_rows && (keys || values)) {
    hipStream_t hs = (hipStream_t)stream;
    const int sid = h->synth_stream, na = h->synth_active;
    s = h->dev(launch_materialize(h->dm, h->ws, sid, na, hs), "read_pseudo/materialize");
    if (s != PROTOKV_OK) return s;
    h->synth_rows = true;
  }
  if (keys) s = copy_out(h, keys, h->ws.pk, n, stream, "read_pseudo");
  if (s == PROTOKV_OK && values) s = copy_out(h, values, h->ws.pv, n, stream, "read_pseudo");
  if (s == PROTOKV_OK && bias) s = copy_out(h, bias, h->ws.pbias, (size_t)h->dm.units * h->dm.K * 4, stream, "read_pseudo");
  return s;
}

protokv_status protokv_state_size(protokv_t h, size_t* bytes) {
  if (!h || !bytes) return PROTOKV_E_INVALID;
  *bytes = state_layout(h->cfg).total;
  return PROTOKV_OK;
}

protokv_status protokv_get_state(protokv_t h, int32_t sid, void* buf, size_t bytes, void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  if (sid < 0 || sid >= h->cfg.num_streams || !buf) return h->fail(PROTOKV_E_INVALID, "get_state: bad stream or buffer");
  const StateLayout sl = state_layout(h->cfg);
  if (bytes != sl.total) return h->fail(PROTOKV_E_INVALID, "get_state: bytes must equal protokv_state_size");
  const StreamState& ss = h->st[sid];
  if (ss.pending) return h->fail(PROTOKV_E_STATE, "get_state: stream has an unfolded eviction");
  const Dims& dm = h->dm;
  const size_t units = dm.units, es = kv_bytes(h->cfg);
  const size_t ring = units * (dm.W + 1) * dm.T * D * es;
  uint8_t* out = (uint8_t*)buf;
  std::memset(out, 0, 256);
  protokv_state_header hd{};
  hd.magic = PROTOKV_STATE_MAGIC;
  hd.version = PROTOKV_STATE_VERSION;
  hd.units = (uint32_t)units;
  hd.capacity = (uint32_t)dm.K;
  hd.tokens_per_frame = (uint32_t)dm.T;
  hd.window_frames = (uint32_t)dm.W;
  hd.kv_bytes = (uint32_t)es;
  hd.codewords = (uint32_t)dm.C;
  hd.warm_tokens = dm.warm_frames > 0 ? (uint32_t)dm.warm_tokens : 0u;
  hd.rotated = h->ws.ring_kr ? 1u : 0u;
  hd.frames = ss.frames;
  hd.evicted_tokens = ss.evicted;
  hd.active_slots = ss.active;
  hd.folds = ss.folds;
  hd.reservoir_rows = ss.rfill;
  hd.off_ring_k = sl.ring_k;
  hd.off_ring_v = sl.ring_v;
  hd.off_bank = sl.bank;
  hd.off_codebooks = sl.codebooks;
  hd.off_reservoir = sl.reservoir;
  hd.off_ring_kr = sl.ring_kr;
  hd.total_bytes = sl.total;
  std::memcpy(out, &hd, sizeof(hd));
  hipStream_t hs = (hipStream_t)stream;
  std::vector<float> cbp(units * 2 * G * CMAX * DP);
  hipError_t e = hipMemcpyAsync(out + sl.ring_k, h->ws.ring_k + sid * ring, ring, hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(out + sl.ring_v, h->ws.ring_v + sid * ring, ring, hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(out + sl.bank, h->ws.bank + (size_t)sid * units * dm.K * ROW, units * dm.K * ROW,
                       hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(cbp.data(), h->ws.codebooks + (size_t)sid * cbp.size(), cbp.size() * 4,
                       hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess && sl.reservoir) {
    const size_t rb = units * 2 * (size_t)dm.warm_tokens * D * 4;
    e = hipMemcpyAsync(out + sl.reservoir, (uint8_t*)h->ws.reservoir + sid * rb, rb, hipMemcpyDeviceToHost, hs);
  }
  if (e == hipSuccess && sl.ring_kr)
    e = hipMemcpyAsync(out + sl.ring_kr, h->ws.ring_kr + sid * ring, ring, hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return h->dev(e, "get_state");
  float* cbo = (float*)(out + sl.codebooks);
  for (size_t blk = 0; blk < units * 2 * G; ++blk)
    std::memcpy(cbo + blk * dm.C * DP, cbp.data() + blk * CMAX * DP, (size_t)dm.C * DP * sizeof(float));
  return PROTOKV_OK;
}

protokv_status protokv_set_state(protokv_t h, int32_t sid, const void* buf, size_t bytes, void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  if (sid < 0 || sid >= h->cfg.num_streams || !buf) return h->fail(PROTOKV_E_INVALID, "set_state: bad stream or buffer");
  const StateLayout sl = state_layout(h->cfg);
  if (bytes != sl.total) return h->fail(PROTOKV_E_INVALID, "set_state: bytes must equal protokv_state_size");
  if (h->st[sid].pending) return h->fail(PROTOKV_E_STATE, "set_state: stream has an unfolded eviction");
  const Dims& dm = h->dm;
  const size_t units = dm.units, es = kv_bytes(h->cfg);
  const uint8_t* in = (const uint8_t*)buf;
  protokv_state_header hd;
  std::memcpy(&hd, in, sizeof(hd));
  auto bad = [&](const char* m) { return h->fail(PROTOKV_E_INVALID, std::string("set_state: ") + m); };
  if (hd.magic != PROTOKV_STATE_MAGIC || hd.version != PROTOKV_STATE_VERSION) return bad("not a state blob");
  if (hd.units != units || hd.capacity != (uint32_t)dm.K || hd.tokens_per_frame != (uint32_t)dm.T ||
      hd.window_frames != (uint32_t)dm.W || hd.kv_bytes != es || hd.codewords != (uint32_t)dm.C ||
      hd.warm_tokens != (dm.warm_frames > 0 ? (uint32_t)dm.warm_tokens : 0u) ||
      hd.rotated != (h->ws.ring_kr ? 1u : 0u))
    return bad("shape differs from the handle's configuration");
  if (hd.off_ring_k != sl.ring_k || hd.off_ring_v != sl.ring_v || hd.off_bank != sl.bank ||
      hd.off_codebooks != sl.codebooks || hd.off_reservoir != sl.reservoir || hd.off_ring_kr != sl.ring_kr ||
      hd.total_bytes != sl.total)
    return bad("section offsets differ from the layout");
  const uint64_t W = (uint64_t)dm.W, T = (uint64_t)dm.T;
  const uint64_t folds = hd.frames > W ? hd.frames - W : 0;
  if ((hd.frames + 1) * T >= (1ull << 31)) return bad("stream position beyond 2^31 tokens");
  if (hd.evicted_tokens != folds * T || (uint64_t)hd.folds != folds)
    return bad("evicted_tokens and folds must follow from frames");
  if (hd.evicted_tokens > PROTOKV_MAX_EVICTED_TOKENS) return bad("evicted_tokens above PROTOKV_MAX_EVICTED_TOKENS");
  if (hd.active_slots < 0 || (uint64_t)hd.active_slots > std::min<uint64_t>(dm.K, hd.evicted_tokens))
    return bad("active_slots outside [0, min(capacity, evicted_tokens)]");
  if (hd.reservoir_rows < 0 || hd.reservoir_rows > (dm.warm_frames > 0 ? dm.warm_tokens : 0))
    return bad("reservoir_rows outside [0, warm_tokens]");
  // bank rows: n > 0 exactly on the active prefix, histogram rows summing to
  // n_res, no counts beyond C codewords, recency within the stream
  const uint8_t* bank = in + sl.bank;
  for (size_t u = 0; u < units; ++u)
    for (int k = 0; k < dm.K; ++k) {
      const uint8_t* row = bank + (u * dm.K + k) * ROW;
      RowMeta m;
      std::memcpy(&m, row + ROW_META, sizeof(m));
      if ((m.n > 0) != (k < hd.active_slots)) return bad("n > 0 must hold exactly on slots [0, active_slots)");
      if (m.n == 0) continue;
      if (m.n_res > hd.evicted_tokens) return bad("n_res above the tokens evicted");
      if (m.tau < 0 || (uint64_t)m.tau >= hd.evicted_tokens + W * T) return bad("tau outside the stream");
      for (int side = 0; side < 2; ++side) {
        const uint32_t* hist = (const uint32_t*)(row + (side ? ROW_HV : ROW_HK));
        for (int g = 0; g < G; ++g) {
          uint64_t tot = 0;
          for (int c = 0; c < CMAX; ++c) {
            if (c >= dm.C && hist[g * CMAX + c]) return bad("histogram count beyond C codewords");
            tot += hist[g * CMAX + c];
          }
          if ((dm.flags & PROTOKV_FLAG_PQ) && tot != m.n_res) return bad("a histogram row does not sum to n_res");
        }
      }
    }
  const float* cbi = (const float*)(in + sl.codebooks);
  for (size_t i = 0; i < units * 2 * G * (size_t)dm.C * DP; ++i)
    if (!std::isfinite(cbi[i])) return bad("non-finite codebook entry");
  std::vector<float> cb = pad_codebooks(cbi, units, dm.C), hn, cmax;
  codebook_tables(cb, dm.C, hn, cmax);
  hipStream_t hs = (hipStream_t)stream;
  const size_t ring = units * (dm.W + 1) * dm.T * D * es;
  hipError_t e = hipMemcpyAsync(h->ws.ring_k + sid * ring, in + sl.ring_k, ring, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(h->ws.ring_v + sid * ring, in + sl.ring_v, ring, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(h->ws.bank + (size_t)sid * units * dm.K * ROW, bank, units * dm.K * ROW,
                       hipMemcpyHostToDevice, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(h->ws.codebooks + (size_t)sid * cb.size(), cb.data(), cb.size() * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(h->ws.cbhn + (size_t)sid * hn.size(), hn.data(), hn.size() * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(h->ws.cbmax + (size_t)sid * cmax.size(), cmax.data(), cmax.size() * 4,
                       hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && sl.reservoir) {
    const size_t rb = units * 2 * (size_t)dm.warm_tokens * D * 4;
    e = hipMemcpyAsync((uint8_t*)h->ws.reservoir + sid * rb, in + sl.reservoir, rb, hipMemcpyHostToDevice, hs);
  }
  if (e == hipSuccess && sl.ring_kr)
    e = hipMemcpyAsync(h->ws.ring_kr + sid * ring, in + sl.ring_kr, ring, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = launch_refresh_all(dm, h->ws, sid, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return h->dev(e, "set_state");
  StreamState& ss = h->st[sid];
  ss.frames = hd.frames;
  ss.evicted = hd.evicted_tokens;
  ss.active = hd.active_slots;
  ss.folds = hd.folds;
  ss.rfill = hd.reservoir_rows;
  ss.pending = false;
  ss.pending_fe = -1;
  if (h->synth_stream == sid) h->synth_stream = -1;
  return PROTOKV_OK;
}

protokv_status protokv_read_pseudo_counts(protokv_t h, int32_t* dst, size_t count, void* stream) {
  if (!h) return PROTOKV_E_INVALID;
  if (!dst) return h->fail(PROTOKV_E_INVALID, "read_pseudo_counts: dst is NULL");
  if (h->synth_stream < 0) return h->fail(PROTOKV_E_STATE, "read_pseudo_counts: no synthesis since the last fold");
  const size_t n = (size_t)h->dm.units * h->dm.K;
  if (count != n) return h->fail(PROTOKV_E_INVALID, "read_pseudo_counts: count must be num_layers*num_kv_heads*capacity");
  if (h->ws.ps_count) return copy_out(h, dst, h->ws.ps_count, n * 4, stream, "read_pseudo_counts");
  for (size_t i = 0; i < n; ++i) dst[i] = (int)(i % h->dm.K) < h->synth_active ? h->dm.S : 0;
  return PROTOKV_OK;
}

protokv_status protokv_profile(protokv_t h, uint32_t kernel_mask) {
  if (!h) return PROTOKV_E_INVALID;
  if (kernel_mask) {
    h->timed.clear();
    h->ev_next = 0;
  }
  h->profile_mask = kernel_mask;
  return PROTOKV_OK;
}

protokv_status protokv_profile_read(protokv_t h, protokv_kernel_times* out) {
  if (!h || !out) return PROTOKV_E_INVALID;
  std::memset(out, 0, sizeof(*out));
  for (const auto& t : h->timed) {
    hipError_t e = hipEventSynchronize(t.b);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, t.a, t.b);
    if (e != hipSuccess) return h->dev(e, "profile_read");
    out->ms[t.id] += ms;
    out->launches[t.id] += 1;
  }
  return PROTOKV_OK;
}

const char* protokv_last_error(protokv_t h) { return h ? h->err.c_str() : g_init_err.c_str(); }

}  // extern "C"
