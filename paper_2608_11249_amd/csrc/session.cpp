// The iterative diffusion compression pipeline (Diffusion-Based Compression
// Pipeline section): every chunk starts masked except for its initial context
// (Initial Context Strategies; none by default) and each pass runs
// forward -> schedule -> CDF -> code -> reveal until no position is masked.
// The entropy schedule computes entropies at every masked row and selects on
// the GPU; the left-to-right block schedules (uniform, progressive) know their
// positions in advance, so only the committed rows go through the LM head.
// Chunks are independent windows; up to `batch` of them share a forward pass,
// and a slot whose chunk is done takes the next one.  Every kernel computes a
// chunk's values independently of the other chunks in the batch, so the
// batch size does not change the output.  Encoding codes on the host from
// each committed symbol's (start, freq); decoding runs the range or rANS
// decoder on the device (decode_symbols), so CDF rows stay in HBM.
#include <cmath>
#include <cstring>

#include "rowstats.h"
#include "runtime.h"

using namespace dlmc;

namespace {

constexpr uint32_t MAGIC = 0x434D4C44u;  // "DLMC" little endian
constexpr uint32_t VERSION = 3;
constexpr size_t FIXED_HEADER = 144;

// Identity of this build's arithmetic: a hash of the library's source code and
// compile flags, set by the build.  The same input coded by two builds whose
// kernels round differently gives different decisions, so a container only
// decodes under the build identity it was made with.
#ifndef DLMC_NUMERICS_ID
#error "DLMC_NUMERICS_ID must be defined by the build (hash of the sources and flags)"
#endif
constexpr uint64_t NUMERICS_ID = DLMC_NUMERICS_ID;

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
  DLMC_CHECK(c.coder == DLMC_CODER_RANGE || c.coder == DLMC_CODER_RANS || c.coder == DLMC_CODER_RANK,
             DLMC_E_INVAL, "unknown coder");
  DLMC_CHECK(c.coder == DLMC_CODER_RANK ? rank_compressor_ok(c.rank_compressor, c.rank_level)
                                        : (c.rank_compressor == 0 && c.rank_level == 0),
             DLMC_E_INVAL, "bad rank compressor / level");
  if (c.coder == DLMC_CODER_RANK) {
    // ranks need no CDF; cdf_bits is unused
  } else if (c.coder == DLMC_CODER_RANGE) {
    DLMC_CHECK(c.coder_bits == 32 || c.coder_bits == 64, DLMC_E_INVAL, "coder_bits must be 32 or 64");
    DLMC_CHECK(c.cdf_bits >= 2 && c.cdf_bits <= c.coder_bits - 16 && (1ll << c.cdf_bits) > m->cfg.vocab,
               DLMC_E_INVAL, "need vocab < 2^cdf_bits and cdf_bits <= coder_bits - 16");
  } else {
    DLMC_CHECK(c.cdf_bits >= 2 && c.cdf_bits <= 31 && (1ll << c.cdf_bits) > m->cfg.vocab,
               DLMC_E_INVAL, "rANS needs vocab < 2^cdf_bits and cdf_bits <= 31");
  }
  DLMC_CHECK(c.schedule >= DLMC_SCHED_ENTROPY && c.schedule <= DLMC_SCHED_PROGRESSIVE, DLMC_E_INVAL,
             "unknown schedule");
  DLMC_CHECK(c.schedule != DLMC_SCHED_UNIFORM || c.blocks >= 1, DLMC_E_INVAL,
             "uniform block schedule needs blocks >= 1");
  DLMC_CHECK(c.schedule != DLMC_SCHED_PROGRESSIVE ||
                 (c.u1 >= 1 && std::isfinite(c.growth) && c.growth > 0.0),
             DLMC_E_INVAL, "progressive schedule needs u1 >= 1 and a finite growth > 0");
  DLMC_CHECK(c.context >= 0 && c.context <= 8192, DLMC_E_INVAL, "context must be in 0..8192");
  DLMC_CHECK(c.context_kind >= DLMC_CONTEXT_CONTIGUOUS && c.context_kind <= DLMC_CONTEXT_ATTENTION,
             DLMC_E_INVAL, "unknown context kind");
  DLMC_CHECK(c.reserved == 0, DLMC_E_INVAL, "reserved field must be 0");
  DLMC_CHECK(c.batch >= 1 && c.batch <= m->cfg.max_batch, DLMC_E_INVAL, "batch must be in 1..max_batch");
  DLMC_CHECK(!std::isnan(c.tau_bits), DLMC_E_INVAL, "tau_bits is NaN");
  DLMC_CHECK((c.flags & ~DLMC_FLAG_CRC) == 0, DLMC_E_INVAL, "unknown flags");
}

// Per-pass commit counts of a left-to-right block schedule over n masked
// positions (Symbol Commitment Schedules, items 1 and 2).
std::vector<int> block_sizes(const dlmc_codec_params& c, int n) {
  std::vector<int> out;
  if (n <= 0) return out;
  if (c.schedule == DLMC_SCHED_UNIFORM) {
    const int K = std::max(1, std::min(c.blocks, n));
    const int u = n / K;
    out.assign(K, u);
    out.back() += n - u * K;
  } else {
    int left = n;
    double g = (double)c.u1;
    while (left > 0) {
      const double r = std::floor(g + 0.5);  // round half up
      const int u = r >= (double)left ? left : std::max(1, (int)r);
      out.push_back(u);
      left -= u;
      g *= c.growth;
    }
  }
  return out;
}

namespace {
// splitmix64 (Steele, Lea and Flood, OOPSLA 2014)
uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
}  // namespace

// Initial-context positions of chunk `chunk` (ascending): the first c, or the
// c positions with the smallest keys splitmix64(splitmix64(seed + chunk) + p)
// (ties by position).
std::vector<int32_t> context_positions(const dlmc_codec_params& c, int T, uint64_t chunk) {
  const int cc = std::min(c.context, T);
  std::vector<int32_t> pos(cc);
  if (cc == 0) return pos;
  if (c.context_kind == DLMC_CONTEXT_CONTIGUOUS) {
    for (int j = 0; j < cc; ++j) pos[j] = j;
    return pos;
  }
  const uint64_t base = splitmix64(c.context_seed + chunk);
  std::vector<std::pair<uint64_t, int32_t>> keys(T);
  for (int p = 0; p < T; ++p) keys[p] = {splitmix64(base + (uint64_t)p), p};
  std::partial_sort(keys.begin(), keys.begin() + cc, keys.end());
  for (int j = 0; j < cc; ++j) pos[j] = keys[j].second;
  std::sort(pos.begin(), pos.end());
  return pos;
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
  (void)hipHostFree(h_state);
  (void)hipHostFree(h_rows);
  (void)hipHostFree(h_selpos);
  (void)hipHostFree(h_selrow);
  (void)hipHostFree(h_nsel_up);
  (void)hipHostFree(h_dslot);
  if (m) {
    m->dfree(d_payload);
    m->dfree(d_dslot);
  }
}

void dlmc_session::assign(int b, uint64_t chunk) {
  const int V = m->cfg.vocab, P = cp.cdf_bits;
  const bool rans = cp.coder == DLMC_CODER_RANS;
  slot_chunk[b] = (int64_t)chunk;
  slot_pass[b] = 0;
  slot_cursor[b] = 0;
  h_base[b] = (int64_t)(chunk * (uint64_t)cp.chunk_len);
  const int c = std::min(cp.context, T);
  auto& cpos = slot_ctx_pos[b];
  auto& csym = slot_ctx_sym[b];
  if (encode) {
    if (cp.context_kind == DLMC_CONTEXT_ATTENTION && c > 0) {
      // two extra passes over this chunk; the c highest scores, ties by position
      std::vector<float> sc;
      m->context_scores(tokens.data() + h_base[b], T, sc);
      std::vector<int32_t> ord(T);
      for (int p = 0; p < T; ++p) ord[p] = p;
      std::stable_sort(ord.begin(), ord.end(), [&](int x, int y) { return sc[x] > sc[y]; });
      cpos.assign(ord.begin(), ord.begin() + c);
      std::sort(cpos.begin(), cpos.end());
    } else {
      cpos = context_positions(cp, T, chunk);
    }
    csym.resize(c);
    for (int j = 0; j < c; ++j) csym[j] = tokens[(size_t)h_base[b] + cpos[j]];
    if (cp.coder == DLMC_CODER_RANK) rk_out[b].clear();
    else if (rans) rencs[b].reset(P);
    else encs[b].reset(cp.coder_bits, P);
  } else {
    const auto& p = payload[chunk];
    DLMC_CHECK(p.size() >= (size_t)6 * c, DLMC_E_CORRUPT, "chunk shorter than its initial context");
    cpos.resize(c);
    csym.resize(c);
    for (int j = 0; j < c; ++j) {
      cpos[j] = get<uint16_t>(p.data(), 2 * (size_t)j);
      csym[j] = (int32_t)get<uint32_t>(p.data(), 2 * (size_t)c + 4 * (size_t)j);
      DLMC_CHECK(cpos[j] < T && (j == 0 || cpos[j] > cpos[j - 1]) && csym[j] >= 0 && csym[j] < V,
                 DLMC_E_CORRUPT, "bad initial context");
      tokens[(size_t)h_base[b] + cpos[j]] = csym[j];
    }
    const uint8_t* data = p.data() + 6 * (size_t)c;
    const size_t len = p.size() - 6 * (size_t)c;
    if (cp.coder == DLMC_CODER_RANK) {
      rk_data[b] = data;
      rk_len[b] = len;
      rk_pos[b] = 0;
    } else {
      // the stream's initial state (host decoder), then the pass-by-pass
      // decoding on the device
      DecSlot& d = h_dslot[b];
      if (rans) {
        if (!rdecs[b].reset(data, len, P)) throw Error(DLMC_E_CORRUPT, "not an rANS stream");
        d.x = rdecs[b].state();
        d.range = 0;
        d.pos = rdecs[b].position();
      } else {
        decs[b].reset(data, len, cp.coder_bits, P);
        d.x = decs[b].code_minus_low();
        d.range = decs[b].range();
        d.pos = decs[b].consumed();
      }
      d.len = len;
      d.off = pl_off[chunk] + 6 * (size_t)c;
      d.live = 1;
      d.pad = 0;
      DLMC_HIP(hipMemcpyAsync(d_dslot + b, &d, sizeof(DecSlot), hipMemcpyHostToDevice, m->stream));
    }
  }
  slot_left[b] = T - c;
  // initial state: [MASK] except the context symbols
  int32_t* hs = h_state + (size_t)b * m->cfg.max_chunk;
  std::fill(hs, hs + T, V);
  for (int j = 0; j < c; ++j) hs[cpos[j]] = csym[j];
  DLMC_HIP(hipMemcpyAsync(m->state + (size_t)b * T, hs, (size_t)T * 4, hipMemcpyHostToDevice, m->stream));
  if (cp.schedule != DLMC_SCHED_ENTROPY) {
    auto& ord = slot_order[b];
    ord.clear();
    for (int p = 0, j = 0; p < T; ++p) {
      if (j < c && cpos[j] == p) {
        ++j;
        continue;
      }
      ord.push_back(p);
    }
  }
}

void dlmc_session::begin_phase() {
  if (phase == 0) {
    // full-length chunks of the range [first_chunk, end_chunk)
    const uint64_t hi = std::min(end_chunk, n_full);
    const uint64_t cnt = hi > first_chunk ? hi - first_chunk : 0;
    B = (int)std::min<uint64_t>((uint64_t)cp.batch, std::max<uint64_t>(cnt, 1));
    T = cp.chunk_len;
    if (cnt == 0) {
      phase = 1;
      begin_phase();
      return;
    }
  } else if (phase == 1) {
    // the final partial chunk, when it exists and lies in the range
    if (n_chunks == n_full || end_chunk < n_chunks) {
      phase = 2;
      return;
    }
    next_chunk = n_full;
    B = 1;
    T = last_len;
  } else {
    return;
  }
  slot_chunk.assign(B, -1);
  slot_left.assign(B, 0);
  slot_pass.assign(B, 0);
  slot_cursor.assign(B, 0);
  slot_ctx_pos.assign(B, {});
  slot_ctx_sym.assign(B, {});
  slot_order.assign(B, {});
  encs.assign(B, RangeEncoder());
  decs.assign(B, RangeDecoder());
  rencs.assign(B, RansEncoder());
  rdecs.assign(B, RansDecoder());
  rk_out.assign(B, {});
  rk_data.assign(B, nullptr);
  rk_len.assign(B, 0);
  rk_pos.assign(B, 0);
  if (cp.schedule != DLMC_SCHED_ENTROPY) blocks = block_sizes(cp, T - std::min(cp.context, T));
  const uint64_t end = phase == 0 ? std::min(end_chunk, n_full) : end_chunk;
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
  if (cp.schedule == DLMC_SCHED_ENTROPY) {
    {
      // the head may leave the logits to selected_logits(); reset even if the forward throws
      struct HeadSlots {
        dlmc_model* m;
        ~HeadSlots() { m->head_slots = 0; }
      } reset{m};
      m->head_slots = B * mm;
      m->forward(m->state, B, T, nullptr, nullptr, nullptr, masked);
    }
    {
      StageTimer t(m, DLMC_STAGE_ENTROPY, m->bf16 ? (double)masked * stat_groups(V) * sizeof(RowStat)
                                                  : (double)masked * V * 4.0);
      m->row_stats(B * T);
    }
    {
      StageTimer t(m, DLMC_STAGE_SELECT, (double)masked * 8.0);
      select_positions(s, m->H, m->rows, m->chunk_off, m->chunk_cnt, B, T, cp.tau_bits, cp.m_min, mm,
                       m->sel_pos, m->sel_row, m->n_sel, m->err);
    }
    m->selected_logits(B, mm);
  } else {
    // the next block of each slot's masked positions, in ascending order
    int r = 0;
    for (int b = 0; b < B; ++b) {
      h_nsel_up[b] = 0;
      if (slot_chunk[b] < 0 || slot_left[b] == 0) continue;
      const int u = blocks[(size_t)slot_pass[b]];
      for (int j = 0; j < u; ++j) {
        const int pos = slot_order[b][(size_t)slot_cursor[b] + j];
        h_selpos[b * mm + j] = pos;
        h_selrow[b * mm + j] = r;
        h_rows[r++] = b * T + pos;
      }
      h_nsel_up[b] = u;
    }
    h_nsel_up[B] = r;
    DLMC_HIP(hipMemcpyAsync(m->rows, h_rows, (size_t)std::max(r, 1) * 4, hipMemcpyHostToDevice, s));
    DLMC_HIP(hipMemcpyAsync(m->n_rows, h_nsel_up + B, 4, hipMemcpyHostToDevice, s));
    DLMC_HIP(hipMemcpyAsync(m->sel_pos, h_selpos, (size_t)B * mm * 4, hipMemcpyHostToDevice, s));
    DLMC_HIP(hipMemcpyAsync(m->sel_row, h_selrow, (size_t)B * mm * 4, hipMemcpyHostToDevice, s));
    DLMC_HIP(hipMemcpyAsync(m->n_sel, h_nsel_up, (size_t)B * 4, hipMemcpyHostToDevice, s));
    m->forward(m->state, B, T, nullptr, nullptr, nullptr, r, true);
    {
      // row statistics (the maximum feeds the CDF) at the committed rows only
      StageTimer t(m, DLMC_STAGE_ENTROPY, m->bf16 ? (double)r * stat_groups(V) * sizeof(RowStat)
                                                  : (double)r * V * 4.0);
      m->row_stats(B * T);
    }
  }
  const bool rank = cp.coder == DLMC_CODER_RANK;
  const size_t cdf_rec = m->prof_recs.size();
  if (!rank) {
    {
      // work (read the row once, write the CDF) is filled in once n_sel is known
      StageTimer t(m, DLMC_STAGE_CDF, 0.0);
      cdf_rows(s, m->logits, m->logit_max(), m->logit_rows(), m->n_sel, B, mm, V, P, m->cdf, nullptr, m->cdf_ws);
    }
    if (encode) {
      StageTimer t(m, DLMC_STAGE_REVEAL, 0.0);
      gather_reveal(s, m->cdf, m->sel_pos, m->n_sel, m->tokens_dev, m->slot_base, m->state, B, T, mm,
                    V, m->sym);
    } else {
      StageTimer t(m, DLMC_STAGE_REVEAL, 0.0);
      decode_symbols(s, m->cdf, m->n_sel, B, mm, V, P, cp.coder_bits, cp.coder == DLMC_CODER_RANS, RANS_L,
                     d_payload, d_dslot, m->dec, m->sym, m->err);
      reveal(s, m->sel_pos, m->n_sel, m->dec, m->state, B, T, mm);
      DLMC_HIP(hipMemcpyAsync(h_dec, m->dec, (size_t)B * mm * 4, hipMemcpyDeviceToHost, s));
      DLMC_HIP(hipMemcpyAsync(h_dslot, d_dslot, (size_t)B * sizeof(DecSlot), hipMemcpyDeviceToHost, s));
    }
  } else if (encode) {
    StageTimer t(m, DLMC_STAGE_REVEAL, 0.0);
    rank_symbols(s, m->logits, m->logit_rows(), m->sel_pos, m->n_sel, m->tokens_dev, m->slot_base,
                 m->state, B, T, mm, V, m->sym);
  }
  DLMC_HIP(hipMemcpyAsync(h_nsel, m->n_sel, (size_t)B * 4, hipMemcpyDeviceToHost, s));
  DLMC_HIP(hipMemcpyAsync(h_pos, m->sel_pos, (size_t)B * mm * 4, hipMemcpyDeviceToHost, s));
  DLMC_HIP(hipMemcpyAsync(h_err, m->err, 4, hipMemcpyDeviceToHost, s));
  if (encode || !rank) DLMC_HIP(hipMemcpyAsync(h_sym, m->sym, (size_t)B * mm * 8, hipMemcpyDeviceToHost, s));
  DLMC_HIP(hipStreamSynchronize(s));
  if (*h_err == 2) throw Error(DLMC_E_CORRUPT, "decoder target out of range");
  if (*h_err) throw Error(DLMC_E_NUMERIC, "non-finite entropy (non-finite logits)");
  if (cdf_rec < m->prof_recs.size() && m->prof_recs[cdf_rec].stage == DLMC_STAGE_CDF) {
    int64_t committed = 0;
    for (int b = 0; b < B; ++b) committed += h_nsel[b];
    m->prof_recs[cdf_rec].work = (double)committed * (8.0 * V + 4.0);
  }
  if (rank && !encode) {
    // this pass's ranks from each slot's stream -> symbols (revealed on the GPU)
    for (int b = 0; b < B; ++b) {
      if (slot_chunk[b] < 0) continue;
      for (int j = 0; j < h_nsel[b]; ++j) {
        uint64_t v = 0;
        int shift = 0;
        for (;;) {
          DLMC_CHECK(rk_pos[b] < rk_len[b] && shift <= 56, DLMC_E_CORRUPT, "rank stream ended early");
          const uint8_t byte = rk_data[b][rk_pos[b]++];
          v |= (uint64_t)(byte & 0x7F) << shift;
          shift += 7;
          if (!(byte & 0x80)) break;
        }
        DLMC_CHECK(v < (uint64_t)V, DLMC_E_CORRUPT, "rank outside the alphabet");
        h_dec[b * mm + j] = (int32_t)v;
      }
    }
    rk_rank.assign(h_dec, h_dec + (size_t)B * mm);
    DLMC_HIP(hipMemcpyAsync(m->dec, h_dec, (size_t)B * mm * 4, hipMemcpyHostToDevice, s));
    {
      StageTimer t(m, DLMC_STAGE_REVEAL, 0.0);
      select_by_rank(s, m->logits, m->logit_rows(), m->sel_pos, m->n_sel, m->dec, m->state, B, T, mm, V);
    }
    DLMC_HIP(hipMemcpyAsync(h_dec, m->dec, (size_t)B * mm * 4, hipMemcpyDeviceToHost, s));
    DLMC_HIP(hipStreamSynchronize(s));
  }

  const size_t row_words = (size_t)V + 1;
  std::vector<int32_t> srow;
  std::vector<float> Hall;
  if (m->trace) {
    // the committed rows' entropies (one copy of the entropies up to the
    // highest committed row), for the per-pass trace
    srow.resize((size_t)B * mm);
    DLMC_HIP(hipMemcpy(srow.data(), m->sel_row, srow.size() * 4, hipMemcpyDeviceToHost));
    int top = -1;
    for (int b = 0; b < B; ++b)
      if (slot_chunk[b] >= 0)
        for (int j = 0; j < h_nsel[b]; ++j) top = std::max(top, srow[(size_t)b * mm + j]);
    Hall.resize((size_t)top + 1);
    if (top >= 0) DLMC_HIP(hipMemcpy(Hall.data(), m->H, Hall.size() * 4, hipMemcpyDeviceToHost));
  }
  std::vector<uint32_t> coded_iv;  // trace: the pass's coded pairs of one slot
  for (int b = 0; b < B; ++b) {
    if (slot_chunk[b] < 0) continue;
    const int ns = h_nsel[b];
    const uint32_t* rows_cdf = nullptr;
    if (!rank && m->trace) {
      // the trace's CDF hash: the only use of the rows on the host
      if (!h_cdf) pinned((void**)&h_cdf, (size_t)mm * row_words * 4);
      DLMC_HIP(hipMemcpy(h_cdf, m->cdf + (size_t)b * mm * row_words, (size_t)ns * row_words * 4,
                         hipMemcpyDeviceToHost));
      rows_cdf = h_cdf;
    }
    const uint64_t chunk = (uint64_t)slot_chunk[b];
    const uint64_t base = chunk * (uint64_t)cp.chunk_len;
    coded_iv.assign((size_t)2 * ns, 0u);
    std::vector<int32_t> syms;  // rank mode: the pass's symbols, for the CDF-free hash
    for (int j = 0; j < ns; ++j) {
      const int pos = h_pos[b * mm + j];
      if (rank) {
        if (encode) {
          uint32_t v = h_sym[2 * (b * mm + j)];
          coded_iv[2 * j] = v;
          coded_iv[2 * j + 1] = h_sym[2 * (b * mm + j) + 1];
          while (v >= 0x80) {
            rk_out[b].push_back((uint8_t)(v | 0x80));
            v >>= 7;
          }
          rk_out[b].push_back((uint8_t)v);
          syms.push_back((int32_t)h_sym[2 * (b * mm + j) + 1]);
        } else {
          tokens[base + pos] = h_dec[b * mm + j];
          syms.push_back(h_dec[b * mm + j]);
          coded_iv[2 * j] = (uint32_t)rk_rank[(size_t)b * mm + j];
          coded_iv[2 * j + 1] = (uint32_t)h_dec[b * mm + j];
        }
      } else if (encode) {
        const uint32_t st = h_sym[2 * (b * mm + j)], fr = h_sym[2 * (b * mm + j) + 1];
        coded_iv[2 * j] = st;
        coded_iv[2 * j + 1] = fr;
        if (cp.coder == DLMC_CODER_RANS) rencs[b].encode(st, fr);
        else encs[b].encode(st, fr);
      } else {
        // decoded on the device
        tokens[base + pos] = h_dec[b * mm + j];
        coded_iv[2 * j] = h_sym[2 * (b * mm + j)];
        coded_iv[2 * j + 1] = h_sym[2 * (b * mm + j) + 1];
      }
    }
    if (m->trace) {
      std::vector<float> hv(ns);
      for (int j = 0; j < ns; ++j) hv[j] = Hall[(size_t)srow[(size_t)b * mm + j]];
      const uint64_t hsh = rank ? fnv1a64(syms.data(), syms.size() * 4)
                                : fnv1a64(rows_cdf, (size_t)ns * row_words * 4);
      m->trace(m->trace_user, encode ? 0 : 1, chunk, slot_pass[b], ns, h_pos + b * mm, hv.data(),
               coded_iv.data(), hsh);
    }
    if (coded) *coded += (uint64_t)ns;
    slot_left[b] -= ns;
    slot_pass[b] += 1;
    slot_cursor[b] += ns;
    DLMC_CHECK(slot_left[b] >= 0 && (ns > 0 || slot_left[b] == 0), DLMC_E_CORRUPT,
               "schedule committed no position");
  }
  ++passes;

  // finished chunks: close their streams and refill their slots
  const uint64_t end = phase == 0 ? std::min(end_chunk, n_full) : end_chunk;
  bool base_changed = false, active = false;
  for (int b = 0; b < B; ++b) {
    if (slot_chunk[b] < 0) continue;
    if (slot_left[b] == 0) {
      const uint64_t chunk = (uint64_t)slot_chunk[b];
      if (encode) {
        // chunk payload: the initial context (u16 positions, u32 symbols), then the coder's bytes
        const auto& cpos = slot_ctx_pos[b];
        const auto& csym = slot_ctx_sym[b];
        const size_t c = cpos.size();
        std::vector<uint8_t> body = cp.coder == DLMC_CODER_RANK   ? std::move(rk_out[b])
                                    : cp.coder == DLMC_CODER_RANS ? rencs[b].finish()
                                                                  : encs[b].finish();
        std::vector<uint8_t> pl(6 * c + body.size());
        for (size_t j = 0; j < c; ++j) {
          put<uint16_t>(pl, 2 * j, (uint16_t)cpos[j]);
          put<uint32_t>(pl, 2 * c + 4 * j, (uint32_t)csym[j]);
        }
        if (!body.empty()) std::memcpy(pl.data() + 6 * c, body.data(), body.size());
        payload[chunk] = std::move(pl);
      } else if (cp.coder == DLMC_CODER_RANS && !(h_dslot[b].pos == h_dslot[b].len && h_dslot[b].x == RANS_L)) {
        throw Error(DLMC_E_CORRUPT, "rANS stream did not end in its initial state");
      } else if (cp.coder == DLMC_CODER_RANK && rk_pos[b] != rk_len[b]) {
        throw Error(DLMC_E_CORRUPT, "rank stream has trailing data");
      }
      if (!encode && (cp.flags & DLMC_FLAG_CRC)) {
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
        if (!encode && !rank) {
          h_dslot[b].live = 0;
          DLMC_HIP(hipMemcpyAsync(d_dslot + b, h_dslot + b, sizeof(DecSlot), hipMemcpyHostToDevice, s));
        }
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

// Container layout (little endian): the 144-byte fixed header below, then
// u64 offsets[count + 1] of the held chunks' payloads inside the payload
// section, then (DLMC_FLAG_CRC) a u32 CRC-32 of each held chunk's tokens, then
// the payload section -- the held chunks' payloads back to back, compressed as
// one block for the symbol ranking back end.  A container holds the chunks
// [first, first + count) of the input's n_chunks; it is complete when it holds
// all of them, and only complete containers decode.
//   0 magic, 4 version, 8 header size, 12 flags, 16 model hash, 24 seed,
//   32 n_tokens, 40 n_chunks, 48.. codec parameters, 116 reserved (0),
//   120 numerics id, 128 first chunk, 136 count
static std::vector<uint8_t> fixed_header(const dlmc_model* m, const dlmc_codec_params& cp, uint64_t n,
                                         uint64_t n_chunks) {
  std::vector<uint8_t> h(FIXED_HEADER, 0);
  put<uint32_t>(h, 0, MAGIC);
  put<uint32_t>(h, 4, VERSION);
  put<uint32_t>(h, 12, (uint32_t)cp.flags);
  put<uint64_t>(h, 16, m->hash());
  put<uint64_t>(h, 24, m->seed);
  put<uint64_t>(h, 32, n);
  put<uint64_t>(h, 40, n_chunks);
  put<int32_t>(h, 48, cp.chunk_len);
  put<int32_t>(h, 52, cp.cdf_bits);
  put<int32_t>(h, 56, cp.coder_bits);
  put<int32_t>(h, 60, cp.m_min);
  put<int32_t>(h, 64, cp.m_max);
  put<float>(h, 68, cp.tau_bits);
  put<int32_t>(h, 72, cp.batch);
  put<int32_t>(h, 76, cp.schedule);
  put<int32_t>(h, 80, cp.blocks);
  put<int32_t>(h, 84, cp.u1);
  put<double>(h, 88, cp.growth);
  put<int32_t>(h, 96, cp.coder);
  put<int32_t>(h, 100, cp.context);
  put<int32_t>(h, 104, cp.context_kind);
  put<int32_t>(h, 108, cp.rank_compressor);
  put<int32_t>(h, 112, cp.rank_level);
  put<uint64_t>(h, 120, NUMERICS_ID);
  return h;
}

// A container from a fixed header (fields 0..127 as above), the held range and
// the held chunks' payloads and CRCs (crc empty unless DLMC_FLAG_CRC).
static std::vector<uint8_t> assemble(std::vector<uint8_t> head, uint64_t first,
                                     const std::vector<std::vector<uint8_t>>& pls,
                                     const std::vector<uint32_t>& crc) {
  const uint64_t cnt = pls.size();
  const bool crc_on = get<uint32_t>(head.data(), 12) & DLMC_FLAG_CRC;
  const int coder = get<int32_t>(head.data(), 96);
  const size_t hdr = FIXED_HEADER + (cnt + 1) * 8 + (crc_on ? cnt * 4 : 0);
  std::vector<uint8_t> section;
  for (const auto& p : pls) section.insert(section.end(), p.begin(), p.end());
  if (coder == DLMC_CODER_RANK)
    section = compress_block(get<int32_t>(head.data(), 108), get<int32_t>(head.data(), 112), section);
  head.resize(hdr + section.size(), 0);
  put<uint32_t>(head, 8, (uint32_t)hdr);
  put<uint64_t>(head, 128, first);
  put<uint64_t>(head, 136, cnt);
  uint64_t off = 0;  // offsets into the (uncompressed) payload section
  for (uint64_t c = 0; c <= cnt; ++c) {
    put<uint64_t>(head, FIXED_HEADER + c * 8, off);
    if (c < cnt) off += pls[c].size();
  }
  if (crc_on)
    for (uint64_t c = 0; c < cnt; ++c) put<uint32_t>(head, FIXED_HEADER + (cnt + 1) * 8 + c * 4, crc[c]);
  if (!section.empty()) std::memcpy(head.data() + hdr, section.data(), section.size());
  return head;
}

std::vector<uint8_t> dlmc_session::container() const {
  std::vector<std::vector<uint8_t>> pls(payload.begin() + first_chunk, payload.begin() + end_chunk);
  std::vector<uint32_t> crc;
  if (cp.flags & DLMC_FLAG_CRC)
    for (uint64_t c = first_chunk; c < end_chunk; ++c) {
      const uint64_t a = c * (uint64_t)cp.chunk_len;
      const uint64_t b = std::min<uint64_t>(n, a + cp.chunk_len);
      crc.push_back(crc32(&tokens[a], (size_t)(b - a) * 4));
    }
  return assemble(fixed_header(m, cp, n, n_chunks), first_chunk, pls, crc);
}

namespace dlmc {

uint64_t numerics_id() { return NUMERICS_ID; }

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
  pinned((void**)&s->h_state, (size_t)m->cfg.max_batch * m->cfg.max_chunk * 4);
  pinned((void**)&s->h_rows, slots * 4);
  pinned((void**)&s->h_selpos, slots * 4);
  pinned((void**)&s->h_selrow, slots * 4);
  pinned((void**)&s->h_nsel_up, ((size_t)m->cfg.max_batch + 1) * 4);
  if (cp.schedule != DLMC_SCHED_ENTROPY) {
    // every block of the full-length and of the final chunk must fit one pass's capacity
    int big = 0;
    for (int len : {s->n_full ? cp.chunk_len : 0, s->last_len})
      for (int u : block_sizes(cp, len - std::min(cp.context, len))) big = std::max(big, u);
    DLMC_CHECK(big <= cp.m_max, DLMC_E_INVAL,
               "a block of the schedule exceeds m_max (" + std::to_string(big) + ")");
  }
  DLMC_HIP(hipMemsetAsync(m->err, 0, 4, m->stream));
}

dlmc_session* make_encoder(dlmc_model* m, const dlmc_codec_params& cp, const int32_t* tokens,
                           uint64_t n, uint64_t first_chunk, uint64_t n_range) {
  DLMC_CHECK(tokens || n == 0, DLMC_E_INVAL, "tokens is NULL");
  for (uint64_t i = 0; i < n; ++i)
    DLMC_CHECK(tokens[i] >= 0 && tokens[i] < m->cfg.vocab, DLMC_E_INVAL,
               "token " + std::to_string(i) + " outside [0, vocab)");
  std::unique_ptr<dlmc_session> s(new dlmc_session());
  s->encode = true;
  s->n = n;
  s->tokens.assign(tokens, tokens + n);
  session_common(s.get(), m, cp);
  if (n_range == UINT64_MAX) n_range = s->n_chunks - std::min(first_chunk, s->n_chunks);
  DLMC_CHECK(first_chunk <= s->n_chunks && n_range <= s->n_chunks - first_chunk &&
                 (n_range >= 1 || s->n_chunks == 0),
             DLMC_E_INVAL, "chunk range outside the input's chunks");
  s->first_chunk = s->next_chunk = first_chunk;
  s->end_chunk = first_chunk + n_range;
  s->payload.assign(s->n_chunks, {});
  m->ensure_tokens(n);
  if (n) DLMC_HIP(hipMemcpyAsync(m->tokens_dev, s->tokens.data(), n * 4, hipMemcpyHostToDevice, m->stream));
  DLMC_HIP(hipStreamSynchronize(m->stream));
  return s.release();
}

void parse_header(const uint8_t* in, uint64_t len, ContainerInfo* ci) {
  DLMC_CHECK(in && len >= FIXED_HEADER, DLMC_E_FORMAT, "container too short");
  DLMC_CHECK(get<uint32_t>(in, 0) == MAGIC, DLMC_E_FORMAT, "bad magic");
  DLMC_CHECK(get<uint32_t>(in, 4) == VERSION, DLMC_E_FORMAT, "unsupported container version");
  DLMC_CHECK(get<uint64_t>(in, 120) == NUMERICS_ID, DLMC_E_FORMAT,
             "container was made by a build with other kernel arithmetic (numerics id mismatch)");
  dlmc_codec_params* cp = &ci->cp;
  *cp = dlmc_codec_params{};
  ci->hdr = get<uint32_t>(in, 8);
  ci->hash = get<uint64_t>(in, 16);
  ci->seed = get<uint64_t>(in, 24);
  ci->n = get<uint64_t>(in, 32);
  ci->n_chunks = get<uint64_t>(in, 40);
  ci->first = get<uint64_t>(in, 128);
  ci->count = get<uint64_t>(in, 136);
  cp->struct_size = sizeof(dlmc_codec_params);
  cp->flags = (int32_t)get<uint32_t>(in, 12);
  cp->chunk_len = get<int32_t>(in, 48);
  cp->cdf_bits = get<int32_t>(in, 52);
  cp->coder_bits = get<int32_t>(in, 56);
  cp->m_min = get<int32_t>(in, 60);
  cp->m_max = get<int32_t>(in, 64);
  cp->tau_bits = get<float>(in, 68);
  cp->batch = get<int32_t>(in, 72);
  cp->schedule = get<int32_t>(in, 76);
  cp->blocks = get<int32_t>(in, 80);
  cp->u1 = get<int32_t>(in, 84);
  cp->growth = get<double>(in, 88);
  cp->coder = get<int32_t>(in, 96);
  cp->context = get<int32_t>(in, 100);
  cp->context_kind = get<int32_t>(in, 104);
  cp->rank_compressor = get<int32_t>(in, 108);
  cp->rank_level = get<int32_t>(in, 112);
  cp->reserved = 0;
  cp->context_seed = 0;  // positions are stored with each chunk
  DLMC_CHECK(cp->chunk_len >= 1, DLMC_E_FORMAT, "bad chunk length");
  DLMC_CHECK(cp->coder == DLMC_CODER_RANGE || cp->coder == DLMC_CODER_RANS || cp->coder == DLMC_CODER_RANK,
             DLMC_E_FORMAT, "unknown coder");
  DLMC_CHECK(cp->coder != DLMC_CODER_RANK || rank_compressor_ok(cp->rank_compressor, cp->rank_level),
             DLMC_E_FORMAT, "bad rank compressor / level");
  // every size below comes from the input: compared by division, or bounded
  // by the buffer length first, so no sum or product can wrap
  const uint64_t cl = (uint64_t)cp->chunk_len;
  DLMC_CHECK(ci->n_chunks == ci->n / cl + (ci->n % cl != 0), DLMC_E_FORMAT, "bad chunk count");
  DLMC_CHECK(ci->first <= ci->n_chunks && ci->count <= ci->n_chunks - ci->first &&
                 (ci->count >= 1 || ci->n_chunks == 0),
             DLMC_E_FORMAT, "bad chunk range");
  const bool crc_on = cp->flags & DLMC_FLAG_CRC;
  // count + 1 offsets (8 bytes each) and, with CRCs, count CRCs (4 bytes) fit
  DLMC_CHECK(len >= FIXED_HEADER + 8 && ci->count <= (len - FIXED_HEADER - 8) / (crc_on ? 12 : 8),
             DLMC_E_FORMAT, "bad header size");
  const uint64_t need = FIXED_HEADER + (ci->count + 1) * 8 + (crc_on ? ci->count * 4 : 0);
  DLMC_CHECK(ci->hdr == need && len >= need, DLMC_E_FORMAT, "bad header size");
  DLMC_CHECK(get<uint64_t>(in, FIXED_HEADER) == 0, DLMC_E_FORMAT, "bad chunk offsets");
  ci->total = get<uint64_t>(in, FIXED_HEADER + ci->count * 8);
}

// The held chunks' payloads of a parsed container (the payload section
// decompressed for the symbol ranking back end), and their CRCs.
static void read_payloads(const uint8_t* in, uint64_t len, const ContainerInfo& ci,
                          std::vector<std::vector<uint8_t>>& pls, std::vector<uint32_t>& crc) {
  const uint64_t nc = ci.count;
  std::vector<uint8_t> unpacked;
  const uint8_t* section = in + ci.hdr;
  if (ci.cp.coder == DLMC_CODER_RANK) {
    // context and varint ranks take at most 11 bytes a token
    DLMC_CHECK(ci.total <= 1024 || (ci.total - 1024) / 16 <= ci.n, DLMC_E_FORMAT, "bad payload size");
    unpacked = decompress_block(ci.cp.rank_compressor, in + ci.hdr, len - ci.hdr, ci.total);
    section = unpacked.data();
  } else {
    DLMC_CHECK(ci.total <= len - ci.hdr, DLMC_E_FORMAT, "bad chunk offsets");
  }
  pls.assign(nc, {});
  crc.assign((ci.cp.flags & DLMC_FLAG_CRC) ? nc : 0, 0u);
  uint64_t prev = 0;
  for (uint64_t c = 0; c < nc; ++c) {
    const uint64_t a = get<uint64_t>(in, FIXED_HEADER + c * 8);
    const uint64_t b = get<uint64_t>(in, FIXED_HEADER + (c + 1) * 8);
    DLMC_CHECK(a == prev && b >= a && b <= ci.total, DLMC_E_FORMAT, "bad chunk offsets");
    pls[c].assign(section + a, section + b);
    prev = b;
    if (ci.cp.flags & DLMC_FLAG_CRC) crc[c] = get<uint32_t>(in, FIXED_HEADER + (nc + 1) * 8 + c * 4);
  }
}

dlmc_session* make_decoder(dlmc_model* m, const uint8_t* in, uint64_t len, int32_t batch) {
  ContainerInfo ci;
  parse_header(in, len, &ci);
  DLMC_CHECK(ci.hash == m->hash(), DLMC_E_FORMAT, "container was made by another model or seed");
  DLMC_CHECK(ci.first == 0 && ci.count == ci.n_chunks, DLMC_E_FORMAT,
             "partial container (a chunk range): merge the parts first");
  dlmc_codec_params cp = ci.cp;
  if (batch > 0) cp.batch = batch;
  cp.batch = std::min(cp.batch, m->cfg.max_batch);
  std::unique_ptr<dlmc_session> s(new dlmc_session());
  s->encode = false;
  s->n = ci.n;
  session_common(s.get(), m, cp);
  s->first_chunk = s->next_chunk = 0;
  s->end_chunk = ci.n_chunks;
  s->tokens.assign(ci.n, 0);
  read_payloads(in, len, ci, s->payload, s->crc);
  if (cp.coder != DLMC_CODER_RANK) {
    // the payload section is the chunks' payloads back to back
    s->pl_off.resize(ci.count + 1);
    for (uint64_t c = 0; c <= ci.count; ++c) s->pl_off[c] = get<uint64_t>(in, FIXED_HEADER + c * 8);
    s->d_payload = (uint8_t*)m->dalloc(ci.total);
    if (ci.total) DLMC_HIP(hipMemcpy(s->d_payload, in + ci.hdr, ci.total, hipMemcpyHostToDevice));
    s->d_dslot = (DecSlot*)m->dalloc((size_t)m->cfg.max_batch * sizeof(DecSlot), true);
    pinned((void**)&s->h_dslot, (size_t)m->cfg.max_batch * sizeof(DecSlot));
    std::memset(s->h_dslot, 0, (size_t)m->cfg.max_batch * sizeof(DecSlot));
  }
  return s.release();
}

std::vector<uint8_t> merge_containers(const uint8_t* const* parts, const uint64_t* lens, int n_parts) {
  DLMC_CHECK(n_parts >= 1 && parts && lens, DLMC_E_INVAL, "no containers to merge");
  std::vector<ContainerInfo> info(n_parts);
  std::vector<int> order(n_parts);
  for (int i = 0; i < n_parts; ++i) {
    DLMC_CHECK(parts[i], DLMC_E_INVAL, "NULL container");
    parse_header(parts[i], lens[i], &info[i]);
    // every header field but the size and the chunk range must agree
    DLMC_CHECK(std::memcmp(parts[i], parts[0], 8) == 0 && std::memcmp(parts[i] + 12, parts[0] + 12, 116) == 0,
               DLMC_E_FORMAT, "containers of different inputs, models or codec parameters");
    order[i] = i;
  }
  std::sort(order.begin(), order.end(), [&](int a, int b) { return info[a].first < info[b].first; });
  std::vector<std::vector<uint8_t>> pls;
  std::vector<uint32_t> crc;
  uint64_t next = 0;
  for (int i : order) {
    DLMC_CHECK(info[i].first == next, DLMC_E_FORMAT, "chunk ranges overlap or leave a gap");
    std::vector<std::vector<uint8_t>> p;
    std::vector<uint32_t> c;
    read_payloads(parts[i], lens[i], info[i], p, c);
    for (auto& x : p) pls.push_back(std::move(x));
    crc.insert(crc.end(), c.begin(), c.end());
    next += info[i].count;
  }
  DLMC_CHECK(next == info[0].n_chunks, DLMC_E_FORMAT, "the containers do not hold every chunk");
  std::vector<uint8_t> head(parts[0], parts[0] + 128);
  head.resize(FIXED_HEADER, 0);
  return assemble(std::move(head), 0, pls, crc);
}

uint64_t encode_bound(const dlmc_codec_params& cp, uint64_t n, uint64_t first, uint64_t count) {
  const uint64_t nc_all = (n + cp.chunk_len - 1) / cp.chunk_len;
  if (first > nc_all) first = nc_all;
  if (count > nc_all - first) count = nc_all - first;
  const uint64_t head = FIXED_HEADER + (count + 1) * 8 + ((cp.flags & DLMC_FLAG_CRC) ? count * 4 : 0);
  uint64_t total = head;
  for (uint64_t c = first; c < first + count; ++c) {
    const uint64_t len = std::min<uint64_t>(cp.chunk_len, n - c * cp.chunk_len);
    const uint64_t ctx = std::min<uint64_t>((uint64_t)cp.context, len);
    const uint64_t coded = len - ctx;
    total += 6 * ctx;
    if (cp.coder == DLMC_CODER_RANK)  // a rank below 2^30 takes at most 5 varint bytes
      total += 5 * coded;
    else if (cp.coder == DLMC_CODER_RANS)  // at most P + 1 bits a symbol for P <= 30, one word for P = 31
      total += 8 + 4 * (cp.cdf_bits <= 30 ? (coded * (cp.cdf_bits + 1) + 31) / 32 : coded);
    else
      total += (coded * (cp.cdf_bits + 1) + 7) / 8 + cp.coder_bits / 8 + 2;
  }
  if (cp.coder == DLMC_CODER_RANK) total += (total - head) / 128 + 1024;  // a compressor's worst case
  return total;
}

}  // namespace dlmc
