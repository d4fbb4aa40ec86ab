// The iterative diffusion compression pipeline (Diffusion-Based Compression
// Pipeline section): every chunk starts fully masked (no initial context) and
// each pass runs forward -> entropy -> schedule -> CDF -> code -> reveal until
// no position is masked.  Chunks are independent windows; up to `batch` of
// them share a forward pass, and a slot whose chunk is done takes the next one.
// Every kernel computes a chunk's values independently of the other chunks in
// the batch, so the batch size does not change the output.
#include <cmath>
#include <cstring>

#include "runtime.h"

using namespace dlmc;

namespace {

constexpr uint32_t MAGIC = 0x434D4C44u;  // "DLMC" little endian
constexpr uint32_t VERSION = 1;
constexpr size_t FIXED_HEADER = 80;

template <typename T>
void put(std::vector<uint8_t>& v, size_t off, T x) {
  std::memcpy(v.data() + off, &x, sizeof(T));
}
template <typename T>
T get(const uint8_t* p, size_t off) {
  T x;
  std::memcpy(&x, p + off, sizeof(T));
  return x;
}

void pinned(void** p, size_t bytes) {
  if (hipHostMalloc(p, std::max<size_t>(bytes, 16), hipHostMallocDefault) != hipSuccess) {
    (void)hipGetLastError();
    throw Error(DLMC_E_NOMEM, "hipHostMalloc failed");
  }
}

}  // namespace

namespace dlmc {

void validate_codec(const dlmc_model* m, const dlmc_codec_params& c) {
  DLMC_CHECK(c.struct_size == sizeof(dlmc_codec_params), DLMC_E_INVAL, "codec struct_size mismatch");
  DLMC_CHECK(c.chunk_len >= 1 && c.chunk_len <= m->cfg.max_chunk, DLMC_E_INVAL,
             "chunk_len must be in 1..max_chunk");
  DLMC_CHECK(c.m_min >= 1 && c.m_max >= c.m_min && c.m_max <= 1024, DLMC_E_INVAL,
             "need 1 <= m_min <= m_max <= 1024");
  DLMC_CHECK(c.coder_bits == 32 || c.coder_bits == 64, DLMC_E_INVAL, "coder_bits must be 32 or 64");
  DLMC_CHECK(c.cdf_bits >= 2 && c.cdf_bits <= c.coder_bits - 16 && c.cdf_bits <= 31 &&
                 (1ll << c.cdf_bits) > m->cfg.vocab,
             DLMC_E_INVAL, "need vocab < 2^cdf_bits and cdf_bits <= coder_bits - 16");
  DLMC_CHECK(c.batch >= 1 && c.batch <= m->cfg.max_batch, DLMC_E_INVAL, "batch must be in 1..max_batch");
  DLMC_CHECK(!std::isnan(c.tau_bits), DLMC_E_INVAL, "tau_bits is NaN");
  DLMC_CHECK((c.flags & ~DLMC_FLAG_CRC) == 0, DLMC_E_INVAL, "unknown flags");
}

}  // namespace dlmc

dlmc_session::~dlmc_session() {
  (void)hipHostFree(h_nsel);
  (void)hipHostFree(h_pos);
  (void)hipHostFree(h_err);
  (void)hipHostFree(h_sym);
  (void)hipHostFree(h_cdf);
  (void)hipHostFree(h_dec);
  (void)hipHostFree(h_base);
}

void dlmc_session::assign(int b, uint64_t chunk) {
  slot_chunk[b] = (int64_t)chunk;
  slot_left[b] = T;
  slot_pass[b] = 0;
  h_base[b] = (int64_t)(chunk * (uint64_t)cp.chunk_len);
  if (encode) {
    encs[b].reset(cp.coder_bits, cp.cdf_bits);
  } else {
    const auto& p = payload[chunk];
    decs[b].reset(p.data(), p.size(), cp.coder_bits, cp.cdf_bits);
  }
  fill_i32(m->stream, m->state + (size_t)b * T, m->cfg.vocab, (size_t)T);
}

void dlmc_session::begin_phase() {
  if (phase == 0) {
    B = (int)std::min<uint64_t>((uint64_t)cp.batch, std::max<uint64_t>(n_full, 1));
    T = cp.chunk_len;
    if (n_full == 0) {
      phase = 1;
      begin_phase();
      return;
    }
  } else if (phase == 1) {
    if (n_chunks == n_full) {
      phase = 2;
      return;
    }
    B = 1;
    T = last_len;
  } else {
    return;
  }
  slot_chunk.assign(B, -1);
  slot_left.assign(B, 0);
  slot_pass.assign(B, 0);
  encs.assign(B, RangeEncoder());
  decs.assign(B, RangeDecoder());
  const uint64_t end = phase == 0 ? n_full : n_chunks;
  for (int b = 0; b < B; ++b) {
    if (next_chunk < end) {
      assign(b, next_chunk++);
    } else {
      h_base[b] = 0;
      fill_i32(m->stream, m->state + (size_t)b * T, 0, (size_t)T);  // nothing masked
    }
  }
  DLMC_HIP(hipMemcpyAsync(m->slot_base, h_base, (size_t)B * 8, hipMemcpyHostToDevice, m->stream));
}

int dlmc_session::step(uint64_t* coded) {
  hipStream_t s = m->stream;
  const int V = m->cfg.vocab, P = cp.cdf_bits, mm = cp.m_max;
  if (!started) {
    started = true;
    begin_phase();
  }
  if (phase == 2) return 1;

  int64_t masked = 0;  // masked positions before this pass (host bookkeeping)
  for (int b = 0; b < B; ++b)
    if (slot_chunk[b] >= 0) masked += slot_left[b];
  m->forward(m->state, B, T, nullptr, nullptr, nullptr, masked);
  {
    StageTimer t(m, DLMC_STAGE_ENTROPY, (double)masked * V * 4.0);
    entropy_rows(s, m->logits, B * T, m->n_rows, V, m->H, m->mx);
  }
  {
    StageTimer t(m, DLMC_STAGE_SELECT, (double)masked * 8.0);
    select_positions(s, m->H, m->rows, m->chunk_off, m->chunk_cnt, B, T, cp.tau_bits, cp.m_min, mm,
                     m->sel_pos, m->sel_row, m->n_sel, m->err);
  }
  const size_t cdf_rec = m->prof_recs.size();
  {
    // work (read the row once, write the CDF) is filled in once n_sel is known
    StageTimer t(m, DLMC_STAGE_CDF, 0.0);
    cdf_rows(s, m->logits, m->mx, m->sel_row, m->n_sel, B, mm, V, P, m->cdf, nullptr, m->cdf_ws);
  }
  if (encode) {
    StageTimer t(m, DLMC_STAGE_REVEAL, 0.0);
    gather_reveal(s, m->cdf, m->sel_pos, m->n_sel, m->tokens_dev, m->slot_base, m->state, B, T, mm,
                  V, m->sym);
  }
  DLMC_HIP(hipMemcpyAsync(h_nsel, m->n_sel, (size_t)B * 4, hipMemcpyDeviceToHost, s));
  DLMC_HIP(hipMemcpyAsync(h_pos, m->sel_pos, (size_t)B * mm * 4, hipMemcpyDeviceToHost, s));
  DLMC_HIP(hipMemcpyAsync(h_err, m->err, 4, hipMemcpyDeviceToHost, s));
  if (encode) DLMC_HIP(hipMemcpyAsync(h_sym, m->sym, (size_t)B * mm * 8, hipMemcpyDeviceToHost, s));
  DLMC_HIP(hipStreamSynchronize(s));
  if (*h_err) throw Error(DLMC_E_NUMERIC, "non-finite entropy (non-finite logits)");
  if (cdf_rec < m->prof_recs.size() && m->prof_recs[cdf_rec].stage == DLMC_STAGE_CDF) {
    int64_t committed = 0;
    for (int b = 0; b < B; ++b) committed += h_nsel[b];
    m->prof_recs[cdf_rec].work = (double)committed * (8.0 * V + 4.0);
  }

  const size_t row_words = (size_t)V + 1;
  std::vector<float> Hsel;
  std::vector<int32_t> srow;
  if (m->trace) {
    // the committed rows' entropies and CDFs, for the per-pass trace
    srow.resize((size_t)B * mm);
    DLMC_HIP(hipMemcpy(srow.data(), m->sel_row, srow.size() * 4, hipMemcpyDeviceToHost));
  }
  bool any_dec = false;
  for (int b = 0; b < B; ++b) {
    if (slot_chunk[b] < 0) continue;
    const int ns = h_nsel[b];
    const uint32_t* rows_cdf = nullptr;
    if (!encode || m->trace) {
      DLMC_HIP(hipMemcpy(h_cdf, m->cdf + (size_t)b * mm * row_words, (size_t)ns * row_words * 4,
                         hipMemcpyDeviceToHost));
      rows_cdf = h_cdf;
    }
    const uint64_t chunk = (uint64_t)slot_chunk[b];
    const uint64_t base = chunk * (uint64_t)cp.chunk_len;
    for (int j = 0; j < ns; ++j) {
      const int pos = h_pos[b * mm + j];
      if (encode) {
        encs[b].encode(h_sym[2 * (b * mm + j)], h_sym[2 * (b * mm + j) + 1]);
      } else {
        const int sym = decs[b].decode(rows_cdf + (size_t)j * row_words, V);
        if (sym < 0) throw Error(DLMC_E_CORRUPT, "range decoder target out of range");
        tokens[base + pos] = sym;
        h_dec[b * mm + j] = sym;
        any_dec = true;
      }
    }
    if (m->trace) {
      std::vector<float> hv(ns);
      for (int j = 0; j < ns; ++j)
        DLMC_HIP(hipMemcpy(&hv[j], m->H + srow[b * mm + j], 4, hipMemcpyDeviceToHost));
      const uint64_t hsh = fnv1a64(rows_cdf, (size_t)ns * row_words * 4);
      m->trace(m->trace_user, encode ? 0 : 1, chunk, slot_pass[b], ns, h_pos + b * mm, hv.data(), hsh);
    }
    if (coded) *coded += (uint64_t)ns;
    slot_left[b] -= ns;
    slot_pass[b] += 1;
    DLMC_CHECK(slot_left[b] >= 0 && (ns > 0 || slot_left[b] == 0), DLMC_E_CORRUPT,
               "schedule committed no position");
  }
  if (!encode && any_dec) {
    DLMC_HIP(hipMemcpyAsync(m->dec, h_dec, (size_t)B * mm * 4, hipMemcpyHostToDevice, s));
    reveal(s, m->sel_pos, m->n_sel, m->dec, m->state, B, T, mm);
  }
  ++passes;

  // finished chunks: close their streams and refill their slots
  const uint64_t end = phase == 0 ? n_full : n_chunks;
  bool base_changed = false, active = false;
  for (int b = 0; b < B; ++b) {
    if (slot_chunk[b] < 0) continue;
    if (slot_left[b] == 0) {
      const uint64_t chunk = (uint64_t)slot_chunk[b];
      if (encode) {
        payload[chunk] = encs[b].finish();
      } else if (cp.flags & DLMC_FLAG_CRC) {
        const uint64_t base = chunk * (uint64_t)cp.chunk_len;
        const int len = phase == 0 ? cp.chunk_len : last_len;
        if (crc32(&tokens[base], (size_t)len * 4) != crc[chunk])
          throw Error(DLMC_E_CORRUPT, "chunk CRC mismatch");
      }
      if (next_chunk < end) {
        assign(b, next_chunk++);
      } else {
        slot_chunk[b] = -1;
        fill_i32(s, m->state + (size_t)b * T, 0, (size_t)T);
      }
      base_changed = true;
    }
    active |= slot_chunk[b] >= 0;
  }
  if (base_changed)
    DLMC_HIP(hipMemcpyAsync(m->slot_base, h_base, (size_t)B * 8, hipMemcpyHostToDevice, s));
  if (!active) {
    phase += 1;
    begin_phase();
  }
  DLMC_HIP(hipStreamSynchronize(s));
  return phase == 2 ? 1 : 0;
}

std::vector<uint8_t> dlmc_session::container() const {
  const bool crc_on = cp.flags & DLMC_FLAG_CRC;
  const size_t hdr = FIXED_HEADER + (n_chunks + 1) * 8 + (crc_on ? n_chunks * 4 : 0);
  size_t total = hdr;
  for (const auto& p : payload) total += p.size();
  std::vector<uint8_t> out(total, 0);
  put<uint32_t>(out, 0, MAGIC);
  put<uint32_t>(out, 4, VERSION);
  put<uint32_t>(out, 8, (uint32_t)hdr);
  put<uint32_t>(out, 12, (uint32_t)cp.flags);
  put<uint64_t>(out, 16, m->hash());
  put<uint64_t>(out, 24, m->seed);
  put<uint64_t>(out, 32, n);
  put<uint64_t>(out, 40, n_chunks);
  put<int32_t>(out, 48, cp.chunk_len);
  put<int32_t>(out, 52, cp.cdf_bits);
  put<int32_t>(out, 56, cp.coder_bits);
  put<int32_t>(out, 60, cp.m_min);
  put<int32_t>(out, 64, cp.m_max);
  put<float>(out, 68, cp.tau_bits);
  put<int32_t>(out, 72, cp.batch);
  uint64_t off = 0;
  for (uint64_t c = 0; c <= n_chunks; ++c) {
    put<uint64_t>(out, FIXED_HEADER + c * 8, off);
    if (c < n_chunks) off += payload[c].size();
  }
  if (crc_on)
    for (uint64_t c = 0; c < n_chunks; ++c) {
      const uint64_t a = c * (uint64_t)cp.chunk_len;
      const uint64_t b = std::min<uint64_t>(n, a + cp.chunk_len);
      put<uint32_t>(out, FIXED_HEADER + (n_chunks + 1) * 8 + c * 4,
                    crc32(&tokens[a], (size_t)(b - a) * 4));
    }
  size_t w = hdr;
  for (const auto& p : payload) {
    if (!p.empty()) std::memcpy(out.data() + w, p.data(), p.size());
    w += p.size();
  }
  return out;
}

namespace dlmc {

static void session_common(dlmc_session* s, dlmc_model* m, const dlmc_codec_params& cp) {
  s->m = m;
  s->cp = cp;
  validate_codec(m, cp);
  m->ensure_sel(cp.m_max);
  s->n_chunks = (s->n + cp.chunk_len - 1) / cp.chunk_len;
  s->n_full = s->n / cp.chunk_len;
  s->last_len = (int)(s->n - s->n_full * cp.chunk_len);
  const size_t slots = (size_t)m->cfg.max_batch * cp.m_max;
  pinned((void**)&s->h_nsel, (size_t)m->cfg.max_batch * 4);
  pinned((void**)&s->h_pos, slots * 4);
  pinned((void**)&s->h_err, 4);
  pinned((void**)&s->h_sym, slots * 8);
  pinned((void**)&s->h_dec, slots * 4);
  pinned((void**)&s->h_base, (size_t)m->cfg.max_batch * 8);
  pinned((void**)&s->h_cdf, (size_t)cp.m_max * ((size_t)m->cfg.vocab + 1) * 4);
  DLMC_HIP(hipMemsetAsync(m->err, 0, 4, m->stream));
}

dlmc_session* make_encoder(dlmc_model* m, const dlmc_codec_params& cp, const int32_t* tokens,
                           uint64_t n) {
  DLMC_CHECK(tokens || n == 0, DLMC_E_INVAL, "tokens is NULL");
  for (uint64_t i = 0; i < n; ++i)
    DLMC_CHECK(tokens[i] >= 0 && tokens[i] < m->cfg.vocab, DLMC_E_INVAL,
               "token " + std::to_string(i) + " outside [0, vocab)");
  std::unique_ptr<dlmc_session> s(new dlmc_session());
  s->encode = true;
  s->n = n;
  s->tokens.assign(tokens, tokens + n);
  session_common(s.get(), m, cp);
  s->payload.assign(s->n_chunks, {});
  m->ensure_tokens(n);
  if (n) DLMC_HIP(hipMemcpyAsync(m->tokens_dev, s->tokens.data(), n * 4, hipMemcpyHostToDevice, m->stream));
  DLMC_HIP(hipStreamSynchronize(m->stream));
  return s.release();
}

void parse_header(const uint8_t* in, uint64_t len, dlmc_codec_params* cp, uint64_t* n,
                  uint64_t* n_chunks, uint64_t* hash, uint64_t* seed, uint32_t* hdr) {
  DLMC_CHECK(in && len >= FIXED_HEADER, DLMC_E_FORMAT, "container too short");
  DLMC_CHECK(get<uint32_t>(in, 0) == MAGIC, DLMC_E_FORMAT, "bad magic");
  DLMC_CHECK(get<uint32_t>(in, 4) == VERSION, DLMC_E_FORMAT, "unsupported container version");
  *hdr = get<uint32_t>(in, 8);
  *hash = get<uint64_t>(in, 16);
  *seed = get<uint64_t>(in, 24);
  *n = get<uint64_t>(in, 32);
  *n_chunks = get<uint64_t>(in, 40);
  cp->struct_size = sizeof(dlmc_codec_params);
  cp->flags = (int32_t)get<uint32_t>(in, 12);
  cp->chunk_len = get<int32_t>(in, 48);
  cp->cdf_bits = get<int32_t>(in, 52);
  cp->coder_bits = get<int32_t>(in, 56);
  cp->m_min = get<int32_t>(in, 60);
  cp->m_max = get<int32_t>(in, 64);
  cp->tau_bits = get<float>(in, 68);
  cp->batch = get<int32_t>(in, 72);
  DLMC_CHECK(cp->chunk_len >= 1, DLMC_E_FORMAT, "bad chunk length");
  DLMC_CHECK(*n_chunks == (*n + cp->chunk_len - 1) / cp->chunk_len, DLMC_E_FORMAT, "bad chunk count");
  const bool crc_on = cp->flags & DLMC_FLAG_CRC;
  const uint64_t need = FIXED_HEADER + (*n_chunks + 1) * 8 + (crc_on ? *n_chunks * 4 : 0);
  DLMC_CHECK(*hdr == need && len >= need, DLMC_E_FORMAT, "bad header size");
}

dlmc_session* make_decoder(dlmc_model* m, const uint8_t* in, uint64_t len, int32_t batch) {
  dlmc_codec_params cp{};
  uint64_t n, nc, hash, seed;
  uint32_t hdr;
  parse_header(in, len, &cp, &n, &nc, &hash, &seed, &hdr);
  DLMC_CHECK(hash == m->hash(), DLMC_E_FORMAT, "container was made by another model or seed");
  if (batch > 0) cp.batch = batch;
  cp.batch = std::min(cp.batch, m->cfg.max_batch);
  std::unique_ptr<dlmc_session> s(new dlmc_session());
  s->encode = false;
  s->n = n;
  session_common(s.get(), m, cp);
  s->tokens.assign(n, 0);
  s->payload.resize(nc);
  s->crc.resize(nc);
  uint64_t prev = 0;
  for (uint64_t c = 0; c < nc; ++c) {
    const uint64_t a = get<uint64_t>(in, FIXED_HEADER + c * 8);
    const uint64_t b = get<uint64_t>(in, FIXED_HEADER + (c + 1) * 8);
    DLMC_CHECK(a == prev && b >= a && hdr + b <= len, DLMC_E_FORMAT, "bad chunk offsets");
    s->payload[c].assign(in + hdr + a, in + hdr + b);
    prev = b;
    if (cp.flags & DLMC_FLAG_CRC) s->crc[c] = get<uint32_t>(in, FIXED_HEADER + (nc + 1) * 8 + c * 4);
  }
  return s.release();
}

uint64_t encode_bound(const dlmc_codec_params& cp, uint64_t n) {
  const uint64_t nc = (n + cp.chunk_len - 1) / cp.chunk_len;
  uint64_t total = FIXED_HEADER + (nc + 1) * 8 + ((cp.flags & DLMC_FLAG_CRC) ? nc * 4 : 0);
  for (uint64_t c = 0; c < nc; ++c) {
    const uint64_t len = std::min<uint64_t>(cp.chunk_len, n - c * cp.chunk_len);
    total += (len * (cp.cdf_bits + 1) + 7) / 8 + cp.coder_bits / 8 + 2;
  }
  return total;
}

}  // namespace dlmc
