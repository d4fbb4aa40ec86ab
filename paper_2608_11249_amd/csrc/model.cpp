// The masked diffusion LM (Definition 3 of the paper) on one GPU: weight
// generation, workspace, and the launch sequence of one forward pass.
#include <cmath>
#include <cstring>

#include "rowstats.h"
#include "runtime.h"

using namespace dlmc;

dlmc_model::~dlmc_model() {
  if (device >= 0) (void)hipSetDevice(device);
  if (stream) (void)hipStreamSynchronize(stream);
  for (auto& r : prof_recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (hipEvent_t e : prof_pool) (void)hipEventDestroy(e);
  for (void* p : allocs) (void)hipFree(p);
  if (own_stream) (void)hipStreamDestroy(own_stream);
}

void* dlmc_model::dalloc(size_t bytes, bool zero) {
  if (bytes == 0) bytes = 16;
  void* p = nullptr;
  if (hipMalloc(&p, bytes) != hipSuccess || !p) {
    (void)hipGetLastError();
    throw Error(DLMC_E_NOMEM, "hipMalloc of " + std::to_string(bytes) + " bytes failed");
  }
  allocs.push_back(p);
  if (zero) DLMC_HIP(hipMemsetAsync(p, 0, bytes, stream));
  return p;
}

void dlmc_model::dfree(void* p) {
  if (!p) return;
  for (auto it = allocs.begin(); it != allocs.end(); ++it)
    if (*it == p) {
      DLMC_HIP(hipStreamSynchronize(stream));
      (void)hipFree(p);
      allocs.erase(it);
      return;
    }
}

void dlmc_model::ensure_sel(int m_max) {
  if (m_max <= sel_cap) return;
  dfree(sel_pos);
  dfree(sel_row);
  dfree(n_sel);
  dfree(dec);
  dfree(cdf);
  dfree(sym);
  dfree(slot_base);
  dfree(cdf_ws);
  dfree(slot_rows);
  dfree(slot_mx);
  const size_t slots = (size_t)cfg.max_batch * m_max;
  sel_pos = (int32_t*)dalloc(slots * 4, true);
  sel_row = (int32_t*)dalloc(slots * 4, true);
  dec = (int32_t*)dalloc(slots * 4, true);
  n_sel = (int32_t*)dalloc((size_t)cfg.max_batch * 4, true);
  cdf = (uint32_t*)dalloc(slots * (size_t)(cfg.vocab + 1) * 4);
  sym = (uint32_t*)dalloc(slots * 8, true);
  slot_base = (int64_t*)dalloc((size_t)cfg.max_batch * 8, true);
  cdf_ws = dalloc(cdf_workspace_bytes(slots, cfg.vocab));
  slot_rows = (int32_t*)dalloc(slots * 4);
  slot_mx = (float*)dalloc(slots * 4, true);
  std::vector<int32_t> iota(slots);
  for (size_t i = 0; i < slots; ++i) iota[i] = (int32_t)i;
  DLMC_HIP(hipMemcpy(slot_rows, iota.data(), slots * 4, hipMemcpyHostToDevice));
  sel_cap = m_max;
}

void dlmc_model::ensure_tokens(size_t n) {
  if (n <= tokens_cap && tokens_dev) return;
  dfree(tokens_dev);
  tokens_dev = (int32_t*)dalloc(std::max<size_t>(n, 1) * 4);
  tokens_cap = n;
}

hipEvent_t dlmc_model::prof_event() {
  if (!prof_pool.empty()) {
    hipEvent_t e = prof_pool.back();
    prof_pool.pop_back();
    return e;
  }
  // timing only: the stream is synchronised before the elapsed times are
  // read, so the events need no system-scope fence (whose L2 writeback would
  // add several microseconds around each timed launch)
  hipEvent_t e;
  DLMC_HIP(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
  return e;
}

void dlmc_model::prof_collect() {
  if (prof_recs.empty()) return;
  DLMC_HIP(hipStreamSynchronize(stream));
  for (auto& r : prof_recs) {
    float ms = 0.0f;
    DLMC_HIP(hipEventElapsedTime(&ms, r.a, r.b));
    prof_ms[r.stage] += ms;
    prof_work[r.stage] += r.work;
    prof_n[r.stage] += 1;
    prof_pool.push_back(r.a);
    prof_pool.push_back(r.b);
  }
  prof_recs.clear();
}

void dlmc_model::prof_reset() {
  prof_collect();
  for (int i = 0; i < DLMC_N_STAGES; ++i) {
    prof_ms[i] = prof_work[i] = 0.0;
    prof_n[i] = 0;
  }
}

namespace dlmc {

uint64_t fnv1a64(const void* data, size_t n, uint64_t h) {
  const uint8_t* p = (const uint8_t*)data;
  for (size_t i = 0; i < n; ++i) {
    h ^= p[i];
    h *= 0x100000001B3ull;
  }
  return h;
}

uint32_t crc32(const void* data, size_t n) {
  static uint32_t table[256];
  static bool init = false;
  if (!init) {
    for (uint32_t i = 0; i < 256; ++i) {
      uint32_t c = i;
      for (int k = 0; k < 8; ++k) c = (c & 1) ? 0xEDB88320u ^ (c >> 1) : c >> 1;
      table[i] = c;
    }
    init = true;
  }
  uint32_t c = 0xFFFFFFFFu;
  const uint8_t* p = (const uint8_t*)data;
  for (size_t i = 0; i < n; ++i) c = table[(c ^ p[i]) & 0xFF] ^ (c >> 8);
  return c ^ 0xFFFFFFFFu;
}

static void validate(const dlmc_model_config& c) {
  DLMC_CHECK(c.struct_size == sizeof(dlmc_model_config), DLMC_E_INVAL, "config struct_size mismatch");
  DLMC_CHECK(c.n_layers >= 0 && c.d_model > 0 && c.n_heads > 0 && c.d_ffn > 0, DLMC_E_INVAL,
             "non-positive model dimension");
  DLMC_CHECK(c.vocab >= 2 && c.vocab < (1 << 30), DLMC_E_INVAL, "vocab out of range");
  DLMC_CHECK(c.d_model % c.n_heads == 0, DLMC_E_INVAL, "d_model must be a multiple of n_heads");
  DLMC_CHECK(c.ffn_kind == DLMC_FFN_GELU || c.ffn_kind == DLMC_FFN_SWIGLU, DLMC_E_INVAL, "ffn_kind");
  DLMC_CHECK(c.norm_kind == DLMC_NORM_LAYER || c.norm_kind == DLMC_NORM_RMS, DLMC_E_INVAL, "norm_kind");
  DLMC_CHECK(c.dtype == DLMC_DTYPE_F32 || c.dtype == DLMC_DTYPE_BF16, DLMC_E_INVAL, "dtype");
  DLMC_CHECK(c.max_chunk >= 1 && c.max_chunk <= 8192, DLMC_E_INVAL, "max_chunk must be in 1..8192");
  DLMC_CHECK(c.max_batch >= 1 && (int64_t)c.max_batch * c.max_chunk <= (1 << 20), DLMC_E_INVAL,
             "max_batch * max_chunk must be in 1..2^20");
  DLMC_CHECK(c.d_model <= 8192, DLMC_E_INVAL, "d_model above 8192");
  const int dh = c.d_model / c.n_heads;
  if (c.dtype == DLMC_DTYPE_BF16) {
    DLMC_CHECK(c.d_model % 128 == 0 && c.d_ffn % 64 == 0, DLMC_E_INVAL,
               "bf16 model needs d_model a multiple of 128 and d_ffn a multiple of 64");
    DLMC_CHECK(dh == 64 || dh == 128, DLMC_E_INVAL, "bf16 model needs head dim 64 or 128");
  } else {
    DLMC_CHECK(c.d_model % 16 == 0 && c.d_ffn % 16 == 0, DLMC_E_INVAL,
               "fp32 model needs d_model and d_ffn multiples of 16");
    DLMC_CHECK(dh == 16 || dh == 32 || dh == 64 || dh == 128, DLMC_E_INVAL,
               "fp32 model needs head dim 16, 32, 64 or 128");
  }
  const int exps[5] = {c.embed_exp, c.attn_exp, c.ffn_in_exp, c.ffn_out_exp, c.head_exp};
  for (int e : exps) DLMC_CHECK(e >= -8 && e <= 60, DLMC_E_INVAL, "weight scale exponent out of range");
  DLMC_CHECK(std::isfinite(c.rope_theta) && c.rope_theta > 1.0f, DLMC_E_INVAL, "rope_theta");
  DLMC_CHECK(std::isfinite(c.norm_eps) && c.norm_eps >= 0.0f, DLMC_E_INVAL, "norm_eps");
}

void create_model(dlmc_model* m, const dlmc_model_config& cfg, uint64_t seed, int device) {
  validate(cfg);
  int ndev = 0;
  DLMC_HIP(hipGetDeviceCount(&ndev));
  DLMC_CHECK(device >= 0 && device < ndev, DLMC_E_INVAL, "no such HIP device");
  m->device = device;
  DLMC_HIP(hipSetDevice(device));
  m->scratch = scratch_address(device);  // looked up once per device, with it current
  DLMC_HIP(hipStreamCreateWithFlags(&m->own_stream, hipStreamNonBlocking));
  m->stream = m->own_stream;
  m->cfg = cfg;
  m->seed = seed;
  m->bf16 = cfg.dtype == DLMC_DTYPE_BF16;
  m->esz = m->bf16 ? 2 : 4;
  const int d = cfg.d_model, F = cfg.d_ffn, V = cfg.vocab, L = cfg.n_layers, H = cfg.n_heads;
  m->dh = d / H;
  const int dh = m->dh, dt = cfg.dtype;
  const bool glu = cfg.ffn_kind == DLMC_FFN_SWIGLU;
  const int nF = glu ? 2 * F : F;
  hipStream_t st = m->stream;

  // every buffer is allocated before any kernel runs, so a model that does
  // not fit fails with E_NOMEM and nothing launched
  // ---- weights
  m->embed = m->dalloc((size_t)(V + 1) * d * m->esz);
  m->head = m->dalloc((size_t)V * d * m->esz);
  for (int l = 0; l < L; ++l) {
    dlmc_model::Layer w{};
    w.wqkv = m->dalloc((size_t)3 * d * d * m->esz);
    w.wo = m->dalloc((size_t)d * d * m->esz);
    w.win = m->dalloc((size_t)nF * d * m->esz);
    w.wout = m->dalloc((size_t)d * F * m->esz);
    m->layers.push_back(w);
  }
  const int half = dh / 2, T = cfg.max_chunk;
  m->rope_cos = (float*)m->dalloc((size_t)T * half * 4);
  m->rope_sin = (float*)m->dalloc((size_t)T * half * 4);

  // ---- workspace
  const size_t R = (size_t)cfg.max_batch * cfg.max_chunk;
  m->max_rows = (int)R;
  m->Tp_max = round_up(cfg.max_chunk, 128);
  const size_t qkv_elems = (size_t)cfg.max_batch * H * m->Tp_max * dh;
  m->x = (float*)m->dalloc(R * d * 4);
  m->h = m->dalloc(R * d * m->esz);
  m->q = m->dalloc(qkv_elems * m->esz);
  m->k = m->dalloc(qkv_elems * m->esz);
  m->vt = m->dalloc(qkv_elems * m->esz);
  m->attn = m->dalloc(R * d * m->esz);
  m->ffn = m->dalloc(R * F * m->esz);
  if (!m->bf16) m->tmp = (float*)m->dalloc(R * std::max(3 * d, nF) * 4);
  m->hm = m->dalloc(R * d * m->esz);
  m->logits = (float*)m->dalloc(R * V * 4);
  if (m->bf16) m->stats = m->dalloc(R * (size_t)stat_groups(V) * sizeof(RowStat));
  m->H = (float*)m->dalloc(R * 4);
  m->mx = (float*)m->dalloc(R * 4);
  m->rows = (int32_t*)m->dalloc(R * 4);
  m->n_rows = (int32_t*)m->dalloc(4);
  m->chunk_off = (int32_t*)m->dalloc((size_t)cfg.max_batch * 4);
  m->chunk_cnt = (int32_t*)m->dalloc((size_t)cfg.max_batch * 4);
  m->state = (int32_t*)m->dalloc(R * 4);
  m->err = (int32_t*)m->dalloc(4);

  // Q, K, V^T padding rows are read (with zero weight) by attention: keep them finite
  DLMC_HIP(hipMemsetAsync(m->q, 0, qkv_elems * m->esz, st));
  DLMC_HIP(hipMemsetAsync(m->k, 0, qkv_elems * m->esz, st));
  DLMC_HIP(hipMemsetAsync(m->vt, 0, qkv_elems * m->esz, st));
  DLMC_HIP(hipMemsetAsync(m->n_rows, 0, 4, st));
  DLMC_HIP(hipMemsetAsync(m->err, 0, 4, st));

  // ---- weight generation
  init_weights(st, m->embed, dt, seed, 1, V + 1, d, cfg.embed_exp, MAP_IDENTITY, 0, dh);
  init_weights(st, m->head, dt, seed, 2, V, d, cfg.head_exp, MAP_IDENTITY, 0, dh);
  const RowMap qk_map = m->bf16 ? MAP_QK_PAIRS : MAP_IDENTITY;
  for (int l = 0; l < L; ++l) {
    const dlmc_model::Layer& w = m->layers[l];
    const int base = 16 + 16 * l;
    init_weights(st, w.wqkv, dt, seed, base + 0, d, d, cfg.attn_exp, qk_map, 0, dh);
    init_weights(st, w.wqkv, dt, seed, base + 1, d, d, cfg.attn_exp, qk_map, d, dh);
    init_weights(st, w.wqkv, dt, seed, base + 2, d, d, cfg.attn_exp, MAP_IDENTITY, 2 * d, dh);
    init_weights(st, w.wo, dt, seed, base + 3, d, d, cfg.attn_exp, MAP_IDENTITY, 0, dh);
    if (glu && m->bf16) {
      init_weights(st, w.win, dt, seed, base + 4, F, d, cfg.ffn_in_exp, MAP_GLU_PAIRS, 0, dh);
      init_weights(st, w.win, dt, seed, base + 5, F, d, cfg.ffn_in_exp, MAP_GLU_PAIRS, 32, dh);
    } else {
      init_weights(st, w.win, dt, seed, base + 4, F, d, cfg.ffn_in_exp, MAP_IDENTITY, 0, dh);
      if (glu) init_weights(st, w.win, dt, seed, base + 5, F, d, cfg.ffn_in_exp, MAP_IDENTITY, F, dh);
    }
    init_weights(st, w.wout, dt, seed, base + 6, d, F, cfg.ffn_out_exp, MAP_IDENTITY, 0, dh);
  }

  // ---- rotary table: angle = t * theta^(-2i/dh), computed in fp64
  std::vector<float> cs((size_t)T * half), sn((size_t)T * half);
  for (int t = 0; t < T; ++t)
    for (int i = 0; i < half; ++i) {
      const double ang = (double)t * std::pow((double)cfg.rope_theta, -2.0 * i / dh);
      cs[(size_t)t * half + i] = (float)std::cos(ang);
      sn[(size_t)t * half + i] = (float)std::sin(ang);
    }
  DLMC_HIP(hipMemcpyAsync(m->rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice, st));
  DLMC_HIP(hipMemcpyAsync(m->rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice, st));
  DLMC_HIP(hipStreamSynchronize(st));
}

}  // namespace dlmc

uint64_t dlmc_model::hash() const {
  const int32_t f[] = {cfg.n_layers,  cfg.d_model,   cfg.n_heads,  cfg.d_ffn,
                       cfg.vocab,     cfg.ffn_kind,  cfg.norm_kind, cfg.dtype,
                       cfg.embed_exp, cfg.attn_exp,  cfg.ffn_in_exp, cfg.ffn_out_exp,
                       cfg.head_exp};
  uint64_t h = fnv1a64(f, sizeof(f));
  uint32_t theta, eps;
  std::memcpy(&theta, &cfg.rope_theta, 4);
  std::memcpy(&eps, &cfg.norm_eps, 4);
  h = fnv1a64(&theta, 4, h);
  h = fnv1a64(&eps, 4, h);
  return fnv1a64(&seed, 8, h);
}

void dlmc_model::forward(const int32_t* st_dev, int B, int T, float* logits_out, int32_t* rows_out,
                         int32_t* n_rows_out, int64_t rows_hint, bool rows_given, float* attn_maps) {
  DLMC_CHECK(B >= 1 && B <= cfg.max_batch && T >= 1 && T <= cfg.max_chunk, DLMC_E_INVAL,
             "batch / chunk length exceed the model's workspace");
  const int d = cfg.d_model, F = cfg.d_ffn, V = cfg.vocab, H = cfg.n_heads;
  const int M = B * T, Tp = round_up(T, 128);
  const bool glu = cfg.ffn_kind == DLMC_FFN_SWIGLU;
  const int nF = glu ? 2 * F : F;
  float* lg = logits_out ? logits_out : logits;
  int32_t* rw = rows_out ? rows_out : rows;
  int32_t* nr = n_rows_out ? n_rows_out : n_rows;
  hipStream_t s = stream;
  const double Md = M, dd = d, es = (double)esz;
  const double head_rows = rows_hint >= 0 ? (double)rows_hint : Md;
  // the one layer whose stages are timed (DLMC_PROFILE_ONE_LAYER), else -1
  const int timed_layer =
      prof && prof_one_layer ? (int)(prof_fwd++ % (uint64_t)layers.size()) : -1;
  prof_gated = false;
  head_deferred = false;

  {
    StageTimer t(this, DLMC_STAGE_EMBED, Md * dd * (es + 4.0));
    dlmc::embed(s, st_dev, this->embed, cfg.dtype, x, M, d, V);
  }
  EpiArgs qkv;
  qkv.q = q;
  qkv.k = k;
  qkv.vt = vt;
  qkv.rope_cos = rope_cos;
  qkv.rope_sin = rope_sin;
  qkv.T = T;
  qkv.Tp = Tp;
  qkv.H = H;
  qkv.dh = dh;
  qkv.d = d;
  EpiArgs resid;
  resid.out = x;
  resid.ldo = d;
  const double norm_bytes = Md * dd * (4.0 + es);
  DLMC_CHECK(!attn_maps || B == 1, DLMC_E_INVAL, "attention maps are taken one chunk at a time");
  // head-averaged attention probabilities of layer l into attn_maps[l] (one
  // S = Q_h K_h^T product per head, softmax added in head order)
  auto attention_map = [&](int l) {
    float* A = attn_maps + (size_t)l * T * T;
    const float scale = 1.0f / std::sqrt((float)dh);
    for (int hd = 0; hd < H; ++hd) {
      EpiArgs e;
      e.out = ctx_S;
      e.ldo = T;
      const size_t off = (size_t)hd * Tp * dh;
      if (bf16)
        gemm_bf16(s, (const bf16_t*)q + off, (const bf16_t*)k + off, T, T, dh, nullptr, EPI_STORE_F32, e);
      else
        gemm_f32(s, (const float*)q + off, (const float*)k + off, T, T, dh, nullptr, EPI_STORE_F32, e);
      softmax_accumulate(s, ctx_S, A, T, scale, 1.0f / H, hd == 0);
    }
  };
  int layer_index = 0;
  for (const Layer& w : layers) {
    prof_gated = timed_layer >= 0 && layer_index != timed_layer;
    {
      StageTimer t(this, DLMC_STAGE_NORM, norm_bytes);
      norm_rows(s, x, h, cfg.dtype, M, d, cfg.norm_kind, cfg.norm_eps, nullptr, nullptr);
    }
    if (bf16) {
      {
        StageTimer t(this, DLMC_STAGE_QKV, 2.0 * Md * 3.0 * dd * dd);
        gemm_bf16(s, (const bf16_t*)h, (const bf16_t*)w.wqkv, M, 3 * d, d, nullptr, EPI_QKV_ROPE, qkv);
      }
      if (attn_maps) attention_map(layer_index);
      {
        StageTimer t(this, DLMC_STAGE_ATTN, 4.0 * B * H * (double)T * T * dh);
        attention_bf16(s, (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)vt, (bf16_t*)attn, B, H, T, Tp, dh);
      }
      {
        StageTimer t(this, DLMC_STAGE_OPROJ, 2.0 * Md * dd * dd);
        gemm_bf16(s, (const bf16_t*)attn, (const bf16_t*)w.wo, M, d, d, nullptr, EPI_RESIDUAL, resid);
      }
    } else {
      EpiArgs t3;
      t3.out = tmp;
      t3.ldo = 3 * d;
      {
        StageTimer t(this, DLMC_STAGE_QKV, 2.0 * Md * 3.0 * dd * dd);
        gemm_f32(s, (const float*)h, (const float*)w.wqkv, M, 3 * d, d, nullptr, EPI_STORE_F32, t3);
        qkv_rope_f32(s, tmp, M, qkv);
      }
      if (attn_maps) attention_map(layer_index);
      {
        StageTimer t(this, DLMC_STAGE_ATTN, 4.0 * B * H * (double)T * T * dh);
        attention_f32(s, (const float*)q, (const float*)k, (const float*)vt, (float*)attn, B, H, T, Tp, dh);
      }
      {
        StageTimer t(this, DLMC_STAGE_OPROJ, 2.0 * Md * dd * dd);
        gemm_f32(s, (const float*)attn, (const float*)w.wo, M, d, d, nullptr, EPI_RESIDUAL, resid);
      }
    }
    {
      StageTimer t(this, DLMC_STAGE_NORM, norm_bytes);
      norm_rows(s, x, h, cfg.dtype, M, d, cfg.norm_kind, cfg.norm_eps, nullptr, nullptr);
    }
    if (bf16) {
      EpiArgs f;
      f.out = ffn;
      f.ldo = F;
      {
        StageTimer t(this, DLMC_STAGE_FFN_IN, 2.0 * Md * nF * dd);
        gemm_bf16(s, (const bf16_t*)h, (const bf16_t*)w.win, M, nF, d, nullptr,
                  glu ? EPI_SWIGLU : EPI_GELU, f);
      }
      {
        StageTimer t(this, DLMC_STAGE_FFN_OUT, 2.0 * Md * dd * F);
        gemm_bf16(s, (const bf16_t*)ffn, (const bf16_t*)w.wout, M, d, F, nullptr, EPI_RESIDUAL, resid);
      }
    } else {
      EpiArgs t2;
      t2.out = tmp;
      t2.ldo = nF;
      {
        StageTimer t(this, DLMC_STAGE_FFN_IN, 2.0 * Md * nF * dd);
        gemm_f32(s, (const float*)h, (const float*)w.win, M, nF, d, nullptr, EPI_STORE_F32, t2);
        ffn_act_f32(s, tmp, (float*)ffn, M, F, cfg.ffn_kind);
      }
      {
        StageTimer t(this, DLMC_STAGE_FFN_OUT, 2.0 * Md * dd * F);
        gemm_f32(s, (const float*)ffn, (const float*)w.wout, M, d, F, nullptr, EPI_RESIDUAL, resid);
      }
    }
    ++layer_index;
  }
  prof_gated = false;
  if (attn_maps) return;  // context passes need no head
  // masked (or given) rows only: compaction, final norm gathered, LM head
  if (!rows_given) {
    StageTimer t(this, DLMC_STAGE_COMPACT, Md * 8.0);
    compact_masked(s, st_dev, B, T, V, rw, nr, chunk_off, chunk_cnt);
  }
  {
    StageTimer t(this, DLMC_STAGE_NORM, head_rows * dd * (4.0 + es));
    norm_rows(s, x, hm, cfg.dtype, M, d, cfg.norm_kind, cfg.norm_eps, rw, nr);
  }
  if (inject_nan) poison_head_input(s, hm, bf16 ? 1 : 0, nr);
  // Deferred logits: when writing the fp32 logits of every masked row would
  // take longer than a second read of the head's weights for the committed
  // rows (about 6 TB/s for the stores, 5 TB/s for the weights, 1 PFLOP/s),
  // the head writes only the entropy statistics and selected_logits()
  // computes the committed rows' logits after the selection.  A row's
  // logits do not depend on the other rows of a launch, so both give the
  // same bits.
  if (bf16 && !logits_out && !rows_given && head_slots > 0 && head_slots <= max_rows &&
      rows_hint > 0 && head_mode != 2) {
    const double Vd = V, store_us = (double)rows_hint * Vd * 4.0 / 6.0e6;
    const double redo_us = Vd * dd * es / 5.0e6 + 2.0 * head_slots * Vd * dd / 1.0e9 + 30.0;
    head_deferred = head_mode == 1 || store_us > redo_us;
  }
  EpiArgs o;
  o.out = head_deferred ? nullptr : lg;
  o.ldo = V;
  o.stats = stats;  // the entropy's group statistics, fused into the head's epilogue
  o.stat_ld = stat_groups(V);
  StageTimer t(this, DLMC_STAGE_HEAD, 2.0 * head_rows * V * dd);
  if (bf16)
    gemm_bf16(s, (const bf16_t*)hm, (const bf16_t*)this->head, M, V, d, nr, EPI_STORE_F32, o,
              rows_hint >= 0 ? (int)rows_hint : -1);
  else
    gemm_f32(s, (const float*)hm, (const float*)this->head, M, V, d, nr, EPI_STORE_F32, o);
}

void dlmc_model::selected_logits(int B, int m_max) {
  if (!head_deferred) return;
  const int d = cfg.d_model, V = cfg.vocab, n = B * m_max;
  // h is free once the forward is done: the committed rows' inputs and row
  // maxima, in slot order (empty slots zero)
  gather_slot_rows(stream, (const bf16_t*)hm, mx, sel_row, n_sel, B, m_max, d, (bf16_t*)h, slot_mx);
  EpiArgs o;
  o.out = logits;
  o.ldo = V;
  StageTimer t(this, DLMC_STAGE_HEAD, 2.0 * n * (double)V * d);
  gemm_bf16(stream, (const bf16_t*)h, (const bf16_t*)head, n, V, d, nullptr, EPI_STORE_F32, o);
}

void dlmc_model::row_stats(int n_max) {
  if (bf16)
    entropy_merge(stream, stats, stat_groups(cfg.vocab), cfg.vocab, n_max, n_rows, H, mx);
  else
    entropy_rows(stream, logits, n_max, n_rows, cfg.vocab, H, mx);
}

void dlmc_model::context_scores(const int32_t* tokens, int T, std::vector<float>& score) {
  DLMC_CHECK(T >= 1 && T <= cfg.max_chunk, DLMC_E_INVAL, "chunk length exceeds the model's workspace");
  const int L = cfg.n_layers, V = cfg.vocab;
  if (T > ctx_T) {
    dfree(ctx_maps);
    dfree(ctx_S);
    dfree(ctx_v);
    dfree(ctx_state);
    ctx_maps = (float*)dalloc((size_t)std::max(L, 1) * T * T * 4);
    ctx_S = (float*)dalloc((size_t)T * T * 4);
    ctx_v = (float*)dalloc((size_t)2 * T * 4);
    ctx_state = (int32_t*)dalloc((size_t)T * 4);
    ctx_T = T;
  }
  score.assign(T, 0.0f);
  std::vector<int32_t> st(T);
  std::vector<float> v(T);
  for (int parity = 0; parity < 2; ++parity) {
    for (int p = 0; p < T; ++p) {
      const bool masked = (p & 1) == parity;
      st[p] = masked ? V : tokens[p];
      v[p] = masked ? 1.0f : 0.0f;
    }
    DLMC_HIP(hipMemcpyAsync(ctx_state, st.data(), (size_t)T * 4, hipMemcpyHostToDevice, stream));
    DLMC_HIP(hipMemcpyAsync(ctx_v, v.data(), (size_t)T * 4, hipMemcpyHostToDevice, stream));
    forward(ctx_state, 1, T, nullptr, nullptr, nullptr, -1, false, ctx_maps);
    // 1_M^T A~_L ... A~_1, last layer first
    float *in = ctx_v, *out = ctx_v + T;
    for (int l = L - 1; l >= 0; --l) {
      rollout_step(stream, ctx_maps + (size_t)l * T * T, in, out, T);
      std::swap(in, out);
    }
    DLMC_HIP(hipMemcpyAsync(v.data(), in, (size_t)T * 4, hipMemcpyDeviceToHost, stream));
    DLMC_HIP(hipStreamSynchronize(stream));
    for (int p = 0; p < T; ++p)
      if ((p & 1) != parity) score[p] = v[p];
  }
}
