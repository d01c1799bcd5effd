// Host driver for the RLC-CSC encoder and decoder, built by the CPU test suite
// with AddressSanitizer and UndefinedBehaviorSanitizer: seeded random matrices
// of many shapes, densities and tile heights go through celty_encode_plan,
// celty_encode (1, 3 and all threads) and celty_decode, and the round trip must
// return the kept, non-zero weights; then the documented error paths.
// Exit status 0 on success (the sanitizers abort on the first error).
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "celty.h"

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next_u64() {   // xorshift64*
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return g_state * 0x2545F4914F6CDD1Dull;
}
double next_unit() { return static_cast<double>(next_u64() >> 11) * (1.0 / 9007199254740992.0); }

// A finite fp16 bit pattern: mostly normal numbers, some subnormals and +-0.
uint16_t random_half() {
  const uint64_t r = next_u64();
  const uint16_t sign = static_cast<uint16_t>((r & 1u) << 15);
  const unsigned kind = static_cast<unsigned>((r >> 1) % 16u);
  if (kind == 0) return sign;                                                        // +-0
  if (kind == 1) return static_cast<uint16_t>(sign | (1u + (r >> 8) % 1023u));        // subnormal
  const uint16_t expo = static_cast<uint16_t>(1u + (r >> 8) % 30u);                   // 1..30: finite
  return static_cast<uint16_t>(sign | (expo << 10) | ((r >> 16) & 0x3FFu));
}

int failures = 0;
void check(bool ok, const char* what, int M, int K, int R) {
  if (!ok) {
    std::fprintf(stderr, "FAIL %s (M=%d K=%d R=%d)\n", what, M, K, R);
    ++failures;
  }
}

void round_trip(int M, int K, int R, double keep, double long_gap_rows, bool with_mask, int stride_pad) {
  const int64_t ldw = K + stride_pad, ldm = K + stride_pad;
  std::vector<uint16_t> W(static_cast<size_t>(M) * ldw, 0x7E00u);   // padding cells hold NaN bits, never read
  std::vector<uint8_t> mask(static_cast<size_t>(M) * ldm, 0xAAu);
  for (int r = 0; r < M; ++r) {
    const bool sparse_row = next_unit() < long_gap_rows;   // rows with long runs of pruned entries
    for (int k = 0; k < K; ++k) {
      W[static_cast<size_t>(r) * ldw + k] = random_half();
      const double p = sparse_row ? keep * 0.05 : keep;
      mask[static_cast<size_t>(r) * ldm + k] = next_unit() < p ? static_cast<uint8_t>(1 + next_u64() % 255) : 0u;
    }
  }
  const uint8_t* mp = with_mask ? mask.data() : nullptr;
  int64_t G = 0, nnz = 0, pad = 0;
  check(celty_encode_plan(W.data(), ldw, mp, ldm, M, K, R, CELTY_LAYOUT_RLC, &G, &nnz, &pad) == CELTY_OK, "plan", M, K, R);
  const int T = (M + R - 1) / R;
  std::vector<uint32_t> gptr(static_cast<size_t>(T) * K + 1);
  // values must be 16-byte aligned: over-allocate and align
  std::vector<uint16_t> vbuf(static_cast<size_t>(8 * G + 8));
  uint16_t* values = reinterpret_cast<uint16_t*>((reinterpret_cast<uintptr_t>(vbuf.data()) + 15u) & ~uintptr_t{15});
  std::vector<uint32_t> runs(static_cast<size_t>(G) + 1);
  std::vector<uint16_t> colmax(static_cast<size_t>(K));
  std::vector<uint16_t> Wd(static_cast<size_t>(M) * K);
  std::vector<uint8_t> md(static_cast<size_t>(M) * K);
  const int thread_counts[3] = {1, 3, 0};
  std::vector<uint16_t> first_values;
  std::vector<uint32_t> first_gptr, first_runs;
  for (int ti = 0; ti < 3; ++ti) {
    celty_rlc_csc enc;
    std::memset(&enc, 0, sizeof(enc));
    check(celty_encode(W.data(), ldw, mp, ldm, M, K, R, CELTY_LAYOUT_RLC, gptr.data(), values, runs.data(),
                       colmax.data(), G, &enc,
                       thread_counts[ti]) == CELTY_OK,
          "encode", M, K, R);
    check(enc.n_groups == G && enc.n_nnz == nnz && enc.n_pad == pad, "header counts", M, K, R);
    if (ti == 0) {
      first_values.assign(values, values + 8 * G);
      first_gptr = gptr;
      first_runs.assign(runs.begin(), runs.begin() + G);
    }
    check((G == 0 || std::memcmp(first_values.data(), values, sizeof(uint16_t) * 8 * G) == 0) && first_gptr == gptr &&
              std::equal(first_runs.begin(), first_runs.end(), runs.begin()),
          "thread-count independence", M, K, R);
    check(celty_decode(&enc, Wd.data(), md.data()) == CELTY_OK, "decode", M, K, R);
    for (int r = 0; r < M; ++r)
      for (int k = 0; k < K; ++k) {
        const uint16_t w = W[static_cast<size_t>(r) * ldw + k];
        const bool kept = (mp == nullptr || mask[static_cast<size_t>(r) * ldm + k] != 0) && (w & 0x7FFFu) != 0;
        const uint16_t want = kept ? w : 0u;
        if (Wd[static_cast<size_t>(r) * K + k] != want || md[static_cast<size_t>(r) * K + k] != (kept ? 1u : 0u)) {
          check(false, "round trip", M, K, R);
          r = M;
          break;
        }
      }
  }
  // a corrupted stream (group pointers not monotone) is rejected
  if (T * K >= 2 && G > 0) {
    celty_rlc_csc enc;
    std::memset(&enc, 0, sizeof(enc));
    celty_encode(W.data(), ldw, mp, ldm, M, K, R, CELTY_LAYOUT_RLC, gptr.data(), values, runs.data(), colmax.data(), G,
                 &enc, 1);
    std::vector<uint32_t> bad(gptr);
    bad[1] = static_cast<uint32_t>(G) + 1u;
    enc.gptr = bad.data();
    check(celty_decode(&enc, Wd.data(), md.data()) == CELTY_EFORMAT, "corrupt gptr rejected", M, K, R);
  }
}

void error_paths() {
  uint16_t w[4] = {0x3C00u, 0, 0x3C00u, 0};
  int64_t G = 0, nnz = 0, pad = 0;
  check(celty_encode_plan(nullptr, 2, nullptr, 2, 2, 2, 1, CELTY_LAYOUT_RLC, &G, &nnz, &pad) == CELTY_EINVAL, "null W", 2, 2, 1);
  check(celty_encode_plan(w, 1, nullptr, 2, 2, 2, 1, CELTY_LAYOUT_RLC, &G, &nnz, &pad) == CELTY_EINVAL, "short stride", 2, 2, 1);
  check(celty_encode_plan(w, 2, nullptr, 2, 2, 2, 0, CELTY_LAYOUT_RLC, &G, &nnz, &pad) == CELTY_EINVAL, "R = 0", 2, 2, 0);
  check(celty_encode_plan(w, 2, nullptr, 2, 2, 2, 1, CELTY_LAYOUT_RLC, nullptr, &nnz, &pad) == CELTY_EINVAL, "null output", 2, 2, 1);
  check(celty_encode_plan(w, 2, nullptr, 2, 2, 2, 1, CELTY_LAYOUT_RLC, &G, &nnz, &pad) == CELTY_OK, "plan ok", 2, 2, 1);
  uint32_t gptr[8];
  alignas(16) uint16_t values[64];
  uint32_t runs[8];
  alignas(4) uint16_t cmax[2];
  celty_rlc_csc enc;
  check(celty_encode(w, 2, nullptr, 2, 2, 2, 1, CELTY_LAYOUT_RLC, gptr, values + 1, runs, cmax, G, &enc, 1) == CELTY_EINVAL,
        "misaligned values", 2, 2, 1);
  check(celty_encode(w, 2, nullptr, 2, 2, 2, 1, CELTY_LAYOUT_RLC, gptr, values, runs, cmax, G + 1, &enc, 1) == CELTY_EINVAL,
        "group count mismatch", 2, 2, 1);
  check(celty_encode(w, 2, nullptr, 2, 2, 2, 1, CELTY_LAYOUT_RLC, gptr, values, runs, cmax, G, &enc, -1) == CELTY_EINVAL,
        "negative thread count", 2, 2, 1);
  check(celty_decode(nullptr, nullptr, nullptr) == CELTY_EINVAL, "decode null", 0, 0, 0);
}

}  // namespace

int main() {
  const struct { int M, K, R; double keep, long_gap; bool mask; int pad; } cases[] = {
      {1, 1, 1, 1.0, 0.0, true, 0},     {1, 1, 1, 0.0, 0.0, true, 0},     {7, 9, 1, 0.5, 0.0, true, 3},
      {64, 64, 16, 0.5, 0.3, true, 0},  {65, 63, 64, 0.3, 0.5, true, 1},  {100, 37, 100, 0.9, 0.0, false, 0},
      {257, 129, 64, 0.05, 0.0, true, 0}, {300, 200, 512, 0.5, 0.2, true, 5}, {1000, 77, 256, 0.1, 0.9, true, 0},
      {129, 1000, 16, 0.8, 0.1, true, 0}, {2048, 64, 2048, 0.02, 0.0, true, 0}, {513, 300, 128, 0.3, 0.3, false, 2},
      {1536, 768, 512, 0.5, 0.1, true, 0},   // enough columns that every worker thread gets a share
  };
  for (const auto& c : cases) round_trip(c.M, c.K, c.R, c.keep, c.long_gap, c.mask, c.pad);
  error_paths();
  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("encoder sanitize driver: ok\n");
  return 0;
}
