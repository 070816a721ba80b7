// Sanitizer driver for the host codec (built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_host_sanitizers.py; CPU only).
//
// For seeded random matrices of many shapes and value distributions it
// builds codebooks of all three container formats (with and without the
// joint limit of the split format's two codes), encodes them into buffers of
// exactly the size the size query reports (any write past them is caught),
// checks that the output does not depend on the thread count and that
// validation accepts it, then damages copies (random bytes and bits of the
// header, metadata and streams, and truncation) and checks that validation
// returns a status without reading out of bounds.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "hufflm.h"

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next() {  // xorshift64*
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return g_state * 0x2545F4914F6CDD1Dull;
}
uint32_t below(uint32_t n) { return (uint32_t)(next() % n); }

// bf16 or float16 bit patterns of one of several value distributions
std::vector<uint16_t> matrix(uint64_t n, int kind) {
  std::vector<uint16_t> w(n);
  for (uint64_t i = 0; i < n; ++i) {
    const uint32_t r = (uint32_t)next();
    switch (kind) {
      case 0: w[i] = (uint16_t)r; break;                                      // every pattern
      case 1: w[i] = (uint16_t)(0x3C00 | (r & 0x807F)); break;                 // one exponent
      case 2: {                                                                // geometric exponent
        int e = 120;
        while ((next() & 1) && e > 1) --e;
        w[i] = (uint16_t)((r & 0x807F) | ((uint32_t)e << 7));
        break;
      }
      case 3: w[i] = (uint16_t)((r & 0x807F) | ((118u + (r >> 16) % 8) << 7)); break;  // a few exponents
      default: w[i] = 0x3F80; break;                                           // constant
    }
  }
  return w;
}

int failures = 0;
#define CHECK(c)                                                     \
  do {                                                               \
    if (!(c)) {                                                      \
      std::fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); \
      ++failures;                                                    \
    }                                                                \
  } while (0)

// Encodes with the given encoder at 1 and 3 threads into exact-size buffers;
// returns the container (empty if the encoder refused the input).
template <class Enc>
std::vector<uint8_t> encode_twice(Enc enc) {
  size_t n = 0;
  if (enc(nullptr, &n, 1u) != HL_OK) return {};
  std::vector<uint8_t> a(n), b(n);
  size_t na = n, nb = n;
  CHECK(enc(a.data(), &na, 1u) == HL_OK && na == n);
  CHECK(enc(b.data(), &nb, 3u) == HL_OK && nb == n);
  CHECK(a == b);
  size_t small = n - 1;
  std::vector<uint8_t> c(small);
  CHECK(enc(c.data(), &small, 1u) == HL_ENOMEM);
  return a;
}

void damage_and_validate(const std::vector<uint8_t>& blob) {
  CHECK(hl_validate(blob.data(), blob.size()) == HL_OK);
  for (int k = 0; k < 24; ++k) {
    std::vector<uint8_t> d = blob;
    const int flips = 1 + (int)below(4);
    for (int f = 0; f < flips; ++f) {
      // mostly the header and metadata, sometimes anywhere
      const size_t lim = below(3) ? std::min<size_t>(d.size(), 4096) : d.size();
      d[below((uint32_t)lim)] ^= (uint8_t)(1u << below(8));
    }
    const hl_status s = hl_validate(d.data(), d.size());
    CHECK(s == HL_OK || s == HL_ECORRUPT);
  }
  for (size_t cut : {size_t(0), size_t(1), size_t(64), size_t(127), size_t(128), blob.size() / 2, blob.size() - 1}) {
    if (cut >= blob.size()) continue;
    std::vector<uint8_t> t(blob.begin(), blob.begin() + (long)cut);  // exact allocation: reads past it are caught
    CHECK(hl_validate(t.data(), t.size()) != HL_OK);
  }
}

}  // namespace

int main(int argc, char** argv) {
  const int cases = argc > 1 ? std::atoi(argv[1]) : 60;
  for (int it = 0; it < cases; ++it) {
    const uint32_t S = 8u << below(4);                       // 8 .. 64
    const uint64_t cols = (uint64_t)S * (1 + below(16));
    const uint64_t rows = 1 + below(200);
    const uint64_t n = rows * cols;
    const int kind = (int)below(5);
    const uint32_t gr = below(2) ? 0u : (1u << below(7));  // default or 1 .. 64 (refused where it does not fit)
    std::vector<uint16_t> w = matrix(n, kind);

    // split format, with and without the joint limit of the two codes
    const uint32_t lmax = 4 + below(12);
    const uint32_t pair_max = below(2) ? 0u : (uint32_t)(8 + below(8));
    hl_codebook cb;
    if (hl_build_codebook(w.data(), n, lmax, pair_max, &cb) == HL_OK) {
      auto blob = encode_twice([&](void* out, size_t* bytes, uint32_t th) {
        return hl_encode(w.data(), rows, cols, &cb, S, gr, th, out, bytes);
      });
      if (!blob.empty()) damage_and_validate(blob);
    }
    // whole exponent
    hl_codebook8 cb8;
    if (hl_build_codebook8(w.data(), n, HL_LMAX8_MIN + below(6), &cb8) == HL_OK) {
      auto blob = encode_twice([&](void* out, size_t* bytes, uint32_t th) {
        return hl_encode8(w.data(), rows, cols, &cb8, S, gr, th, out, bytes);
      });
      if (!blob.empty()) damage_and_validate(blob);
    }
    // float16 {1,5,5,5}
    hl_codebook16 cb16;
    if (hl_build_codebook16(w.data(), n, HL_LMAX16_MIN + below(8), &cb16) == HL_OK) {
      auto blob = encode_twice([&](void* out, size_t* bytes, uint32_t th) {
        return hl_encode16(w.data(), rows, cols, &cb16, S, gr, th, out, bytes);
      });
      if (!blob.empty()) damage_and_validate(blob);
    }
  }
  // argument errors
  hl_codebook cb;
  uint16_t one = 0x3F80;
  CHECK(hl_build_codebook(nullptr, 1, 12, 11, &cb) == HL_EINVAL);
  CHECK(hl_build_codebook(&one, 0, 12, 11, &cb) == HL_EINVAL);
  CHECK(hl_build_codebook(&one, 1, 3, 0, &cb) == HL_EINVAL);
  CHECK(hl_validate(nullptr, 0) != HL_OK);
  std::printf("host_fuzz: %d cases, %d failures\n", cases, failures);
  return failures ? 1 : 0;
}
