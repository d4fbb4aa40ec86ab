// Block compression of the symbol-ranking payloads (Experimental Methodology:
// varint ranks compressed by a general-purpose compressor).  zlib is linked;
// liblzma (xz container, CRC-64 check) and libzstd are loaded at run time
// through their public C entry points, so the library still loads on hosts
// without them -- choosing a missing compressor is an error.
#include <dlfcn.h>
#include <zlib.h>

#include <cstring>
#include <mutex>

#include "runtime.h"

namespace dlmc {
namespace {

// liblzma: lzma_ret is an enum (LZMA_OK 0, LZMA_STREAM_END 1), lzma_check too
// (LZMA_CHECK_CRC64 4); the allocator argument may be NULL.
using lzma_easy_buffer_encode_fn = int (*)(uint32_t preset, int check, const void* allocator,
                                           const uint8_t* in, size_t in_size, uint8_t* out,
                                           size_t* out_pos, size_t out_size);
using lzma_stream_buffer_decode_fn = int (*)(uint64_t* memlimit, uint32_t flags, const void* allocator,
                                             const uint8_t* in, size_t* in_pos, size_t in_size,
                                             uint8_t* out, size_t* out_pos, size_t out_size);
using lzma_stream_buffer_bound_fn = size_t (*)(size_t uncompressed_size);
// libzstd
using zstd_compress_fn = size_t (*)(void* dst, size_t cap, const void* src, size_t n, int level);
using zstd_decompress_fn = size_t (*)(void* dst, size_t cap, const void* src, size_t n);
using zstd_bound_fn = size_t (*)(size_t n);
using zstd_is_error_fn = unsigned (*)(size_t code);

struct Lzma {
  lzma_easy_buffer_encode_fn enc = nullptr;
  lzma_stream_buffer_decode_fn dec = nullptr;
  lzma_stream_buffer_bound_fn bound = nullptr;
};
struct Zstd {
  zstd_compress_fn enc = nullptr;
  zstd_decompress_fn dec = nullptr;
  zstd_bound_fn bound = nullptr;
  zstd_is_error_fn is_error = nullptr;
};

void* open_first(std::initializer_list<const char*> names) {
  for (const char* n : names)
    if (void* h = dlopen(n, RTLD_NOW | RTLD_LOCAL)) return h;
  return nullptr;
}

const Lzma& lzma() {
  static Lzma L;
  static std::once_flag once;
  std::call_once(once, [] {
    if (void* h = open_first({"liblzma.so.5", "liblzma.so"})) {
      L.enc = (lzma_easy_buffer_encode_fn)dlsym(h, "lzma_easy_buffer_encode");
      L.dec = (lzma_stream_buffer_decode_fn)dlsym(h, "lzma_stream_buffer_decode");
      L.bound = (lzma_stream_buffer_bound_fn)dlsym(h, "lzma_stream_buffer_bound");
    }
  });
  DLMC_CHECK(L.enc && L.dec && L.bound, DLMC_E_INVAL, "liblzma is not available on this host");
  return L;
}

const Zstd& zstd() {
  static Zstd Z;
  static std::once_flag once;
  std::call_once(once, [] {
    if (void* h = open_first({"libzstd.so.1", "libzstd.so"})) {
      Z.enc = (zstd_compress_fn)dlsym(h, "ZSTD_compress");
      Z.dec = (zstd_decompress_fn)dlsym(h, "ZSTD_decompress");
      Z.bound = (zstd_bound_fn)dlsym(h, "ZSTD_compressBound");
      Z.is_error = (zstd_is_error_fn)dlsym(h, "ZSTD_isError");
    }
  });
  DLMC_CHECK(Z.enc && Z.dec && Z.bound && Z.is_error, DLMC_E_INVAL,
             "libzstd is not available on this host");
  return Z;
}

}  // namespace

bool rank_compressor_ok(int kind, int level) {
  switch (kind) {
    case DLMC_RANKC_NONE: return level == 0;
    case DLMC_RANKC_ZLIB: return level >= 0 && level <= 9;
    case DLMC_RANKC_LZMA: return level >= 0 && level <= 9;
    case DLMC_RANKC_ZSTD: return level >= 1 && level <= 22;
    default: return false;
  }
}

std::vector<uint8_t> compress_block(int kind, int level, const std::vector<uint8_t>& in) {
  std::vector<uint8_t> out;
  if (kind == DLMC_RANKC_NONE) return in;
  if (kind == DLMC_RANKC_ZLIB) {
    uLongf n = compressBound((uLong)in.size());
    out.resize(n);
    DLMC_CHECK(compress2(out.data(), &n, in.data(), (uLong)in.size(), level) == Z_OK, DLMC_E_NOMEM,
               "zlib compression failed");
    out.resize(n);
  } else if (kind == DLMC_RANKC_LZMA) {
    const Lzma& L = lzma();
    out.resize(L.bound(in.size()));
    size_t pos = 0;
    DLMC_CHECK(L.enc((uint32_t)level, 4, nullptr, in.data(), in.size(), out.data(), &pos, out.size()) == 0,
               DLMC_E_NOMEM, "lzma compression failed");
    out.resize(pos);
  } else {
    const Zstd& Z = zstd();
    out.resize(Z.bound(in.size()));
    const size_t n = Z.enc(out.data(), out.size(), in.data(), in.size(), level);
    DLMC_CHECK(!Z.is_error(n), DLMC_E_NOMEM, "zstd compression failed");
    out.resize(n);
  }
  return out;
}

std::vector<uint8_t> decompress_block(int kind, const uint8_t* in, size_t len, size_t expect) {
  std::vector<uint8_t> out(expect);
  if (kind == DLMC_RANKC_NONE) {
    DLMC_CHECK(len == expect, DLMC_E_FORMAT, "payload size mismatch");
    if (len) std::memcpy(out.data(), in, len);
  } else if (kind == DLMC_RANKC_ZLIB) {
    uLongf n = (uLongf)expect;
    DLMC_CHECK(uncompress(out.data(), &n, in, (uLong)len) == Z_OK && n == expect, DLMC_E_CORRUPT,
               "zlib payload does not decompress to its recorded size");
  } else if (kind == DLMC_RANKC_LZMA) {
    const Lzma& L = lzma();
    uint64_t memlimit = UINT64_MAX;
    size_t ip = 0, op = 0;
    DLMC_CHECK(L.dec(&memlimit, 0, nullptr, in, &ip, len, out.data(), &op, out.size()) == 0 &&
                   ip == len && op == expect,
               DLMC_E_CORRUPT, "lzma payload does not decompress to its recorded size");
  } else if (kind == DLMC_RANKC_ZSTD) {
    const Zstd& Z = zstd();
    const size_t n = Z.dec(out.data(), out.size(), in, len);
    DLMC_CHECK(!Z.is_error(n) && n == expect, DLMC_E_CORRUPT,
               "zstd payload does not decompress to its recorded size");
  } else {
    throw Error(DLMC_E_FORMAT, "unknown rank compressor");
  }
  return out;
}

}  // namespace dlmc
