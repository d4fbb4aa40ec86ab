// extern "C" entry points of libdlmc.so: argument checks, exception to
// status conversion, thread-local error text.
#include <cstring>
#include <new>
#include <string>

#include "runtime.h"

using namespace dlmc;

namespace dlmc {
dlmc_session* make_encoder(dlmc_model* m, const dlmc_codec_params& cp, const int32_t* tokens,
                           uint64_t n, uint64_t first_chunk, uint64_t n_range);
dlmc_session* make_decoder(dlmc_model* m, const uint8_t* in, uint64_t len, int32_t batch);
}  // namespace dlmc

namespace {

thread_local std::string g_last_error;

template <typename F>
dlmc_status guard(F&& f) {
  try {
    f();
    return DLMC_OK;
  } catch (const Error& e) {
    g_last_error = e.what();
    return e.code;
  } catch (const std::bad_alloc&) {
    g_last_error = "host allocation failed";
    return DLMC_E_NOMEM;
  } catch (const std::exception& e) {
    g_last_error = e.what();
    return DLMC_E_INVAL;
  }
}

void use(dlmc_model* m) {
  DLMC_CHECK(m, DLMC_E_INVAL, "model is NULL");
  DLMC_HIP(hipSetDevice(m->device));
}

// Device buffers of one call, freed when it returns or throws.
struct DevBufs {
  std::vector<void*> held;
  template <typename T>
  T* alloc(size_t bytes) {
    void* q = nullptr;
    if (hipMalloc(&q, std::max<size_t>(bytes, 16)) != hipSuccess || !q) {
      (void)hipGetLastError();
      throw Error(DLMC_E_NOMEM, "hipMalloc of " + std::to_string(bytes) + " bytes failed");
    }
    held.push_back(q);
    return (T*)q;
  }
  DevBufs() = default;
  DevBufs(const DevBufs&) = delete;
  DevBufs& operator=(const DevBufs&) = delete;
  ~DevBufs() {
    for (void* q : held) (void)hipFree(q);  // hipFree waits for the device
  }
};

dlmc_status write_out(const std::vector<uint8_t>& bytes, uint8_t* out, uint64_t cap,
                      uint64_t* out_len) {
  if (out_len) *out_len = bytes.size();
  if (!out || cap < bytes.size()) {
    g_last_error = "output buffer too small: need " + std::to_string(bytes.size()) + " bytes";
    return DLMC_E_BUFFER;
  }
  std::memcpy(out, bytes.data(), bytes.size());
  return DLMC_OK;
}

}  // namespace

extern "C" {

dlmc_status dlmc_model_create(const dlmc_model_config* cfg, uint64_t seed, int32_t device,
                              dlmc_model** out) {
  return guard([&] {
    DLMC_CHECK(cfg && out, DLMC_E_INVAL, "NULL argument");
    *out = nullptr;
    dlmc_model* m = new dlmc_model();
    try {
      create_model(m, *cfg, seed, device);
    } catch (...) {
      delete m;
      throw;
    }
    *out = m;
  });
}

void dlmc_model_destroy(dlmc_model* model) { delete model; }

dlmc_status dlmc_set_stream(dlmc_model* m, void* hip_stream) {
  return guard([&] {
    use(m);
    DLMC_HIP(hipStreamSynchronize(m->stream));
    m->stream = hip_stream ? (hipStream_t)hip_stream : m->own_stream;
  });
}

dlmc_status dlmc_encode_bound(const dlmc_model* m, const dlmc_codec_params* codec,
                              uint64_t n_tokens, uint64_t* bytes) {
  return guard([&] {
    DLMC_CHECK(m && codec && bytes, DLMC_E_INVAL, "NULL argument");
    validate_codec(m, *codec);
    *bytes = encode_bound(*codec, n_tokens, 0, UINT64_MAX);
  });
}

dlmc_status dlmc_encode_range_bound(const dlmc_model* m, const dlmc_codec_params* codec,
                                    uint64_t n_tokens, uint64_t first_chunk, uint64_t n_chunks,
                                    uint64_t* bytes) {
  return guard([&] {
    DLMC_CHECK(m && codec && bytes, DLMC_E_INVAL, "NULL argument");
    validate_codec(m, *codec);
    *bytes = encode_bound(*codec, n_tokens, first_chunk, n_chunks);
  });
}

dlmc_status dlmc_encoder_begin(dlmc_model* m, const dlmc_codec_params* codec,
                               const int32_t* tokens, uint64_t n, dlmc_session** out) {
  return guard([&] {
    use(m);
    DLMC_CHECK(codec && out, DLMC_E_INVAL, "NULL argument");
    *out = make_encoder(m, *codec, tokens, n, 0, UINT64_MAX);
  });
}

dlmc_status dlmc_encoder_step(dlmc_session* s, int32_t* done, uint64_t* coded) {
  return guard([&] {
    DLMC_CHECK(s && s->encode, DLMC_E_INVAL, "not an encoder session");
    use(s->m);
    const int d = s->step(coded);
    if (done) *done = d;
  });
}

dlmc_status dlmc_encoder_finish(dlmc_session* s, uint8_t* out, uint64_t cap, uint64_t* out_len) {
  dlmc_status st = guard([&] {
    DLMC_CHECK(s && s->encode, DLMC_E_INVAL, "not an encoder session");
    use(s->m);
    while (!s->step(nullptr)) {
    }
  });
  if (st != DLMC_OK) return st;
  return write_out(s->container(), out, cap, out_len);
}

void dlmc_session_destroy(dlmc_session* s) { delete s; }

dlmc_status dlmc_encode(dlmc_model* m, const dlmc_codec_params* codec, const int32_t* tokens,
                        uint64_t n, uint8_t* out, uint64_t cap, uint64_t* out_len) {
  dlmc_session* s = nullptr;
  dlmc_status st = dlmc_encoder_begin(m, codec, tokens, n, &s);
  if (st != DLMC_OK) return st;
  st = dlmc_encoder_finish(s, out, cap, out_len);
  delete s;
  return st;
}

dlmc_status dlmc_encode_range(dlmc_model* m, const dlmc_codec_params* codec, const int32_t* tokens,
                              uint64_t n, uint64_t first_chunk, uint64_t n_chunks, uint8_t* out,
                              uint64_t cap, uint64_t* out_len) {
  dlmc_session* s = nullptr;
  dlmc_status st = guard([&] {
    use(m);
    DLMC_CHECK(codec, DLMC_E_INVAL, "NULL argument");
    s = make_encoder(m, *codec, tokens, n, first_chunk, n_chunks);
  });
  if (st != DLMC_OK) return st;
  st = dlmc_encoder_finish(s, out, cap, out_len);
  delete s;
  return st;
}

dlmc_status dlmc_merge(const uint8_t* const* parts, const uint64_t* lens, int32_t n_parts,
                       uint8_t* out, uint64_t cap, uint64_t* out_len) {
  std::vector<uint8_t> bytes;
  dlmc_status st = guard([&] { bytes = merge_containers(parts, lens, n_parts); });
  if (st != DLMC_OK) return st;
  return write_out(bytes, out, cap, out_len);
}

dlmc_status dlmc_numerics_id(uint64_t* id) {
  return guard([&] {
    DLMC_CHECK(id, DLMC_E_INVAL, "NULL argument");
    *id = numerics_id();
  });
}

dlmc_status dlmc_decode_size(const uint8_t* in, uint64_t len, uint64_t* n_tokens) {
  return guard([&] {
    DLMC_CHECK(n_tokens, DLMC_E_INVAL, "NULL argument");
    ContainerInfo ci;
    parse_header(in, len, &ci);
    *n_tokens = ci.n;
  });
}

dlmc_status dlmc_decode(dlmc_model* m, const uint8_t* in, uint64_t len, int32_t batch,
                        int32_t* tokens, uint64_t cap, uint64_t* n) {
  dlmc_session* s = nullptr;
  dlmc_status st = guard([&] {
    use(m);
    // the output size is checked from the header before any allocation
    ContainerInfo ci;
    parse_header(in, len, &ci);
    if (n) *n = ci.n;
    if (!tokens || cap < ci.n)
      throw Error(DLMC_E_BUFFER, "token buffer too small: need " + std::to_string(ci.n));
    s = make_decoder(m, in, len, batch);
    while (!s->step(nullptr)) {
    }
    if (s->n) std::memcpy(tokens, s->tokens.data(), s->n * 4);
  });
  delete s;
  return st;
}

dlmc_status dlmc_set_trace(dlmc_model* m, dlmc_trace_fn fn, void* user) {
  return guard([&] {
    DLMC_CHECK(m, DLMC_E_INVAL, "model is NULL");
    m->trace = fn;
    m->trace_user = user;
  });
}

dlmc_status dlmc_test_inject_nonfinite(dlmc_model* m, int32_t on) {
  return guard([&] {
    DLMC_CHECK(m, DLMC_E_INVAL, "model is NULL");
    m->inject_nan = on != 0;
  });
}

dlmc_status dlmc_test_head_logits(dlmc_model* m, int32_t mode) {
  return guard([&] {
    DLMC_CHECK(m, DLMC_E_INVAL, "model is NULL");
    DLMC_CHECK(mode >= 0 && mode <= 2, DLMC_E_INVAL, "mode must be 0, 1 or 2");
    m->head_mode = mode;
  });
}

dlmc_status dlmc_test_gemm_tiles(int32_t M, int32_t N, int32_t K, int32_t epi, int32_t d_model,
                                 int32_t* kind, int32_t* split) {
  return guard([&] {
    DLMC_CHECK(kind && split, DLMC_E_INVAL, "NULL argument");
    DLMC_CHECK(M >= 1 && N >= 1 && K >= 64 && K % 64 == 0 && epi >= 0 && epi <= 4, DLMC_E_INVAL,
               "sizes or epilogue the bf16 GEMM does not take");
    DLMC_CHECK((epi != EPI_QKV_ROPE && epi != EPI_SWIGLU) || N % 128 == 0, DLMC_E_INVAL,
               "paired epilogue needs N % 128 == 0");
    const GemmTiles t = gemm_bf16_tiles(M, N, K, (EpiKind)epi, d_model, -1);
    *kind = t.kind;
    *split = t.split;
  });
}

dlmc_status dlmc_forward_logits(dlmc_model* m, const int32_t* state, int32_t B, int32_t T,
                                float* logits, int32_t* rows, int32_t* n_rows) {
  return guard([&] {
    use(m);
    DLMC_CHECK(state && logits && rows && n_rows, DLMC_E_INVAL, "NULL device pointer");
    m->forward(state, B, T, logits, rows, n_rows);
    DLMC_HIP(hipStreamSynchronize(m->stream));
  });
}

dlmc_status dlmc_entropy_cdf(dlmc_model* m, const float* logits, int32_t n_rows, int32_t cdf_bits,
                             float* entropy_bits, float* row_max, uint32_t* g, uint32_t* cdf) {
  return guard([&] {
    use(m);
    DLMC_CHECK(logits && entropy_bits && row_max && n_rows >= 0, DLMC_E_INVAL, "bad argument");
    const int V = m->cfg.vocab;
    hipStream_t s = m->stream;
    if (cdf) {
      DLMC_CHECK(cdf_bits >= 2 && cdf_bits <= 31 && (1ll << cdf_bits) > V, DLMC_E_INVAL,
                 "cdf_bits must be in 2..31 with 2^cdf_bits > vocab");
      DLMC_CHECK(n_rows <= 65535, DLMC_E_INVAL, "at most 65535 CDF rows per call");
    }
    entropy_rows(s, logits, n_rows, nullptr, V, entropy_bits, row_max);
    if (cdf && n_rows > 0) {
      // every row committed: one "chunk" per row, n_sel = 1
      DevBufs bufs;
      int32_t* sel_row = bufs.alloc<int32_t>((size_t)n_rows * 4);
      int32_t* n_sel = bufs.alloc<int32_t>((size_t)n_rows * 4);
      void* ws = bufs.alloc<void>(cdf_workspace_bytes(n_rows, V));
      std::vector<int32_t> idx(n_rows), one(n_rows, 1);
      for (int i = 0; i < n_rows; ++i) idx[i] = i;
      DLMC_HIP(hipMemcpyAsync(sel_row, idx.data(), idx.size() * 4, hipMemcpyHostToDevice, s));
      DLMC_HIP(hipMemcpyAsync(n_sel, one.data(), one.size() * 4, hipMemcpyHostToDevice, s));
      cdf_rows(s, logits, row_max, sel_row, n_sel, n_rows, 1, V, cdf_bits, cdf, g, ws);
      DLMC_HIP(hipStreamSynchronize(s));
    }
    DLMC_HIP(hipStreamSynchronize(s));
  });
}

dlmc_status dlmc_entropy_cdf_noalloc(dlmc_model* m, const float* logits, int32_t n_rows,
                                     int32_t cdf_bits, float* entropy_bits, float* row_max,
                                     uint32_t* g, uint32_t* cdf) {
  return guard([&] {
    use(m);
    DLMC_CHECK(logits && entropy_bits && row_max && n_rows >= 0, DLMC_E_INVAL, "bad argument");
    const int V = m->cfg.vocab;
    hipStream_t s = m->stream;
    // the scratch holds sel_row[n] and n_sel[n], then (256-byte aligned) the
    // CDF segment partials
    const size_t ws_off = ((size_t)n_rows * 8 + 255) & ~(size_t)255;
    const size_t need = cdf ? ws_off + cdf_workspace_bytes((size_t)n_rows, V) : 0;
    if (cdf) {
      DLMC_CHECK(cdf_bits >= 2 && cdf_bits <= 31 && (1ll << cdf_bits) > V, DLMC_E_INVAL,
                 "cdf_bits must be in 2..31 with 2^cdf_bits > vocab");
      DLMC_CHECK(n_rows <= 65535, DLMC_E_INVAL, "at most 65535 CDF rows per call");
      DLMC_CHECK(need <= SCRATCH_BYTES, DLMC_E_INVAL,
                 "n_rows needs " + std::to_string(need) + " bytes of scratch; the static scratch holds " +
                     std::to_string(SCRATCH_BYTES));
    }
    DLMC_CHECK(m->scratch, DLMC_E_DEVICE, "no static scratch on this device");
    entropy_rows(s, logits, n_rows, nullptr, V, entropy_bits, row_max);
    if (cdf && n_rows > 0) {
      uint8_t* base = (uint8_t*)m->scratch;
      int32_t* sel_row = (int32_t*)base;
      int32_t* n_sel = sel_row + n_rows;
      void* ws = base + ws_off;
      fill_row_slots(s, sel_row, n_sel, n_rows);
      cdf_rows(s, logits, row_max, sel_row, n_sel, n_rows, 1, V, cdf_bits, cdf, g, ws);
    }
    DLMC_HIP(hipStreamSynchronize(s));
  });
}

dlmc_status dlmc_select(dlmc_model* m, const float* H, const int32_t* rows, int32_t n_rows,
                        int32_t B, int32_t T, float tau_bits, int32_t m_min, int32_t m_max,
                        int32_t* sel_pos, int32_t* sel_row, int32_t* n_sel) {
  return guard([&] {
    use(m);
    DLMC_CHECK(H && rows && sel_pos && sel_row && n_sel, DLMC_E_INVAL, "NULL device pointer");
    DLMC_CHECK(B >= 1 && B <= m->cfg.max_batch && T >= 1 && n_rows >= 0 && n_rows <= B * T,
               DLMC_E_INVAL, "bad batch shape");
    hipStream_t s = m->stream;
    // chunk segments of the caller's row list (ascending flat indices)
    std::vector<int32_t> hrows(n_rows), off(B), cnt(B, 0);
    if (n_rows) DLMC_HIP(hipMemcpyAsync(hrows.data(), rows, (size_t)n_rows * 4, hipMemcpyDeviceToHost, s));
    DLMC_HIP(hipStreamSynchronize(s));
    int i = 0;
    for (int b = 0; b < B; ++b) {
      off[b] = i;
      while (i < n_rows && hrows[i] < (b + 1) * T) ++i;
      cnt[b] = i - off[b];
    }
    DLMC_HIP(hipMemcpyAsync(m->chunk_off, off.data(), (size_t)B * 4, hipMemcpyHostToDevice, s));
    DLMC_HIP(hipMemcpyAsync(m->chunk_cnt, cnt.data(), (size_t)B * 4, hipMemcpyHostToDevice, s));
    DLMC_HIP(hipMemsetAsync(m->err, 0, 4, s));
    select_positions(s, H, rows, m->chunk_off, m->chunk_cnt, B, T, tau_bits, m_min, m_max, sel_pos,
                     sel_row, n_sel, m->err);
    int32_t err = 0;
    DLMC_HIP(hipMemcpyAsync(&err, m->err, 4, hipMemcpyDeviceToHost, s));
    DLMC_HIP(hipStreamSynchronize(s));
    if (err) throw Error(DLMC_E_NUMERIC, "non-finite entropy");
  });
}

dlmc_status dlmc_weight_copy(dlmc_model* m, int32_t tensor_id, void* dst, uint64_t bytes) {
  return guard([&] {
    use(m);
    DLMC_CHECK(dst, DLMC_E_INVAL, "NULL destination");
    const auto& c = m->cfg;
    const int d = c.d_model, F = c.d_ffn, V = c.vocab, dh = m->dh;
    const bool glu = c.ffn_kind == DLMC_FFN_SWIGLU;
    const void* base = nullptr;
    int rows = 0, cols = d, row_off = 0, map = MAP_IDENTITY;
    if (tensor_id == 1) {
      base = m->embed;
      rows = V + 1;
    } else if (tensor_id == 2) {
      base = m->head;
      rows = V;
    } else {
      const int l = (tensor_id - 16) / 16, kind = (tensor_id - 16) % 16;
      DLMC_CHECK(tensor_id >= 16 && l < c.n_layers && kind <= 6 && (kind != 5 || glu),
                 DLMC_E_INVAL, "no such tensor");
      const auto& w = m->layers[l];
      switch (kind) {
        case 0: case 1: case 2:
          base = w.wqkv; rows = d; row_off = kind * d;
          map = (kind < 2 && m->bf16) ? MAP_QK_PAIRS : MAP_IDENTITY;
          break;
        case 3: base = w.wo; rows = d; break;
        case 4: case 5:
          base = w.win; rows = F;
          if (glu && m->bf16) { map = MAP_GLU_PAIRS; row_off = kind == 5 ? 32 : 0; }
          else row_off = kind == 5 ? F : 0;
          break;
        default: base = w.wout; rows = d; cols = F; break;
      }
    }
    const size_t row_bytes = (size_t)cols * m->esz;
    DLMC_CHECK(bytes == (size_t)rows * row_bytes, DLMC_E_INVAL, "destination size mismatch");
    DLMC_HIP(hipStreamSynchronize(m->stream));
    for (int r = 0; r < rows; ++r) {
      int dr = r;
      if (map == MAP_QK_PAIRS) {
        const int h = r / dh, w = r % dh, half = dh / 2, p = w < half ? w : w - half;
        dr = h * dh + (2 * (p / 32) + (w < half ? 0 : 1)) * 32 + p % 32;
      } else if (map == MAP_GLU_PAIRS) {
        dr = (r / 32) * 64 + r % 32;
      }
      DLMC_HIP(hipMemcpy((uint8_t*)dst + r * row_bytes,
                         (const uint8_t*)base + (size_t)(dr + row_off) * row_bytes, row_bytes,
                         hipMemcpyDeviceToHost));
    }
  });
}

dlmc_status dlmc_profile_enable(dlmc_model* m, uint32_t stage_mask) {
  return guard([&] {
    use(m);
    m->prof_reset();
    m->prof = stage_mask & DLMC_PROFILE_ALL;
    m->prof_one_layer = (stage_mask & DLMC_PROFILE_ONE_LAYER) != 0;
    m->prof_fwd = 0;
  });
}

dlmc_status dlmc_profile_read(dlmc_model* m, int32_t stage, double* ms_total, uint64_t* launches,
                              double* work) {
  return guard([&] {
    use(m);
    DLMC_CHECK(stage >= 0 && stage < DLMC_N_STAGES, DLMC_E_INVAL, "no such stage");
    m->prof_collect();
    if (ms_total) *ms_total = m->prof_ms[stage];
    if (launches) *launches = m->prof_n[stage];
    if (work) *work = m->prof_work[stage];
  });
}

namespace {
// one "chunk" of length 1 per row: slot i commits position 0 of row i
struct RowSlots {
  DevBufs bufs;
  int32_t *sel_row = nullptr, *sel_pos = nullptr, *n_sel = nullptr, *state = nullptr;
  int64_t* base = nullptr;
  uint32_t* pairs = nullptr;
  explicit RowSlots(int n, hipStream_t s) {
    sel_row = bufs.alloc<int32_t>((size_t)n * 4);
    sel_pos = bufs.alloc<int32_t>((size_t)n * 4);
    n_sel = bufs.alloc<int32_t>((size_t)n * 4);
    state = bufs.alloc<int32_t>((size_t)n * 4);
    base = bufs.alloc<int64_t>((size_t)n * 8);
    pairs = bufs.alloc<uint32_t>((size_t)n * 8);
    std::vector<int32_t> idx(n), zero(n, 0), one(n, 1);
    std::vector<int64_t> b(n);
    for (int i = 0; i < n; ++i) idx[i] = i, b[i] = i;
    DLMC_HIP(hipMemcpyAsync(sel_row, idx.data(), (size_t)n * 4, hipMemcpyHostToDevice, s));
    DLMC_HIP(hipMemcpyAsync(sel_pos, zero.data(), (size_t)n * 4, hipMemcpyHostToDevice, s));
    DLMC_HIP(hipMemcpyAsync(n_sel, one.data(), (size_t)n * 4, hipMemcpyHostToDevice, s));
    DLMC_HIP(hipMemcpyAsync(base, b.data(), (size_t)n * 8, hipMemcpyHostToDevice, s));
    DLMC_HIP(hipStreamSynchronize(s));
  }
};
}  // namespace

dlmc_status dlmc_context_scores(dlmc_model* m, const int32_t* tokens, int32_t T, float* scores) {
  return guard([&] {
    use(m);
    DLMC_CHECK(tokens && scores, DLMC_E_INVAL, "NULL argument");
    DLMC_CHECK(T >= 1 && T <= m->cfg.max_chunk, DLMC_E_INVAL, "T must be in 1..max_chunk");
    for (int i = 0; i < T; ++i)
      DLMC_CHECK(tokens[i] >= 0 && tokens[i] < m->cfg.vocab, DLMC_E_INVAL, "token outside [0, vocab)");
    std::vector<float> sc;
    m->context_scores(tokens, T, sc);
    std::memcpy(scores, sc.data(), (size_t)T * 4);
  });
}

dlmc_status dlmc_rank_rows(dlmc_model* m, const float* logits, int32_t n_rows, const int32_t* sym,
                           int32_t* rank) {
  return guard([&] {
    use(m);
    DLMC_CHECK(n_rows >= 0 && n_rows <= 65535, DLMC_E_INVAL, "n_rows must be in 0..65535");
    if (n_rows == 0) return;
    DLMC_CHECK(logits && sym && rank, DLMC_E_INVAL, "NULL argument");
    hipStream_t s = m->stream;
    RowSlots r(n_rows, s);
    rank_symbols(s, logits, r.sel_row, r.sel_pos, r.n_sel, sym, r.base, r.state, n_rows, 1, 1,
                 m->cfg.vocab, r.pairs);
    DLMC_HIP(hipMemcpy2DAsync(rank, 4, r.pairs, 8, 4, n_rows, hipMemcpyDeviceToDevice, s));
    DLMC_HIP(hipStreamSynchronize(s));
  });
}

dlmc_status dlmc_select_rank_rows(dlmc_model* m, const float* logits, int32_t n_rows,
                                  const int32_t* rank, int32_t* sym) {
  return guard([&] {
    use(m);
    DLMC_CHECK(n_rows >= 0 && n_rows <= 65535, DLMC_E_INVAL, "n_rows must be in 0..65535");
    if (n_rows == 0) return;
    DLMC_CHECK(logits && sym && rank, DLMC_E_INVAL, "NULL argument");
    hipStream_t s = m->stream;
    RowSlots r(n_rows, s);
    std::vector<int32_t> h(n_rows);
    DLMC_HIP(hipMemcpy(h.data(), rank, (size_t)n_rows * 4, hipMemcpyDeviceToHost));
    for (int32_t v : h) DLMC_CHECK(v >= 0 && v < m->cfg.vocab, DLMC_E_INVAL, "rank outside the alphabet");
    DLMC_HIP(hipMemcpyAsync(sym, rank, (size_t)n_rows * 4, hipMemcpyDeviceToDevice, s));
    select_by_rank(s, logits, r.sel_row, r.sel_pos, r.n_sel, sym, r.state, n_rows, 1, 1, m->cfg.vocab);
    DLMC_HIP(hipStreamSynchronize(s));
  });
}

dlmc_status dlmc_rc_encode(const uint32_t* start, const uint32_t* freq, uint64_t n,
                           int32_t cdf_bits, int32_t coder_bits, uint8_t* out, uint64_t cap,
                           uint64_t* out_len) {
  std::vector<uint8_t> bytes;
  dlmc_status st = guard([&] {
    DLMC_CHECK((coder_bits == 32 || coder_bits == 64) && cdf_bits >= 1 && cdf_bits <= coder_bits - 16,
               DLMC_E_INVAL, "unsupported coder width / precision");
    DLMC_CHECK(n == 0 || (start && freq), DLMC_E_INVAL, "NULL argument");
    RangeEncoder enc(coder_bits, cdf_bits);
    for (uint64_t i = 0; i < n; ++i) {
      DLMC_CHECK(freq[i] >= 1 && (uint64_t)start[i] + freq[i] <= (1ull << cdf_bits), DLMC_E_INVAL,
                 "bad symbol interval");
      enc.encode(start[i], freq[i]);
    }
    bytes = enc.finish();
  });
  if (st != DLMC_OK) return st;
  return write_out(bytes, out, cap, out_len);
}

dlmc_status dlmc_rc_decode(const uint8_t* in, uint64_t len, const uint32_t* cdf, uint64_t n,
                           int32_t V, int32_t cdf_bits, int32_t coder_bits, int32_t* sym) {
  return guard([&] {
    DLMC_CHECK((coder_bits == 32 || coder_bits == 64) && cdf_bits >= 1 && cdf_bits <= coder_bits - 16,
               DLMC_E_INVAL, "unsupported coder width / precision");
    DLMC_CHECK(n == 0 || (in && cdf && sym && V >= 1), DLMC_E_INVAL, "NULL argument");
    RangeDecoder dec(in, len, coder_bits, cdf_bits);
    for (uint64_t i = 0; i < n; ++i) {
      const int s = dec.decode(cdf + i * ((uint64_t)V + 1), V);
      if (s < 0) throw Error(DLMC_E_CORRUPT, "range decoder target out of range");
      sym[i] = s;
    }
  });
}

dlmc_status dlmc_rans_encode(const uint32_t* start, const uint32_t* freq, uint64_t n,
                             int32_t cdf_bits, uint8_t* out, uint64_t cap, uint64_t* out_len) {
  std::vector<uint8_t> bytes;
  dlmc_status st = guard([&] {
    DLMC_CHECK(cdf_bits >= 1 && cdf_bits <= 31, DLMC_E_INVAL, "rANS needs 1 <= cdf_bits <= 31");
    DLMC_CHECK(n == 0 || (start && freq), DLMC_E_INVAL, "NULL argument");
    RansEncoder enc;
    enc.reset(cdf_bits);
    for (uint64_t i = 0; i < n; ++i) {
      DLMC_CHECK(freq[i] >= 1 && (uint64_t)start[i] + freq[i] <= (1ull << cdf_bits), DLMC_E_INVAL,
                 "bad symbol interval");
      enc.encode(start[i], freq[i]);
    }
    bytes = enc.finish();
  });
  if (st != DLMC_OK) return st;
  return write_out(bytes, out, cap, out_len);
}

dlmc_status dlmc_rans_decode(const uint8_t* in, uint64_t len, const uint32_t* cdf, uint64_t n,
                             int32_t V, int32_t cdf_bits, int32_t* sym) {
  return guard([&] {
    DLMC_CHECK(cdf_bits >= 1 && cdf_bits <= 31, DLMC_E_INVAL, "rANS needs 1 <= cdf_bits <= 31");
    DLMC_CHECK(n == 0 || (cdf && sym && V >= 1), DLMC_E_INVAL, "NULL argument");
    DLMC_CHECK(in || len == 0, DLMC_E_INVAL, "NULL stream");
    RansDecoder dec;
    if (!dec.reset(in, len, cdf_bits)) throw Error(DLMC_E_CORRUPT, "not an rANS stream");
    for (uint64_t i = 0; i < n; ++i) {
      const int s = dec.decode(cdf + i * ((uint64_t)V + 1), V);
      if (s < 0) throw Error(DLMC_E_CORRUPT, "rANS stream corrupt");
      sym[i] = s;
    }
    if (!dec.done()) throw Error(DLMC_E_CORRUPT, "rANS stream did not end in its initial state");
  });
}

const char* dlmc_status_string(dlmc_status s) {
  switch (s) {
    case DLMC_OK: return "ok";
    case DLMC_E_INVAL: return "invalid argument";
    case DLMC_E_NOMEM: return "out of memory";
    case DLMC_E_DEVICE: return "HIP device error";
    case DLMC_E_FORMAT: return "bad container format";
    case DLMC_E_CORRUPT: return "corrupt bitstream";
    case DLMC_E_BUFFER: return "buffer too small";
    case DLMC_E_NUMERIC: return "non-finite values";
    default: return "unknown status";
  }
}

const char* dlmc_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
