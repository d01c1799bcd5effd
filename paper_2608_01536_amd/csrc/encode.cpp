// Host RLC-CSC encoder and decoder (offline packing, Section 3.2).
//
// Work is split into items (row tile t, block of columns); an item walks the
// rows of its tile in memory order, keeping per-column state, so W and the
// mask are read row-major and contiguously.  Segments of one item are
// contiguous in the tile-major layout, so items never write the same bytes
// and the output does not depend on the thread count.
//
// Three layouts of the rows: 4-bit runs (the paper's); 16-bit row offsets
// within the tile (no padding entries, a decode-free form); and the RLC
// entries of each segment in lane-interleaved order within chunks of up to
// 64 groups (Section 4.2), produced by permuting each item's segments after
// the RLC fill.

#include <algorithm>
#include <atomic>
#include <cstring>
#include <new>
#include <thread>
#include <vector>

#include "celty.h"

namespace {

constexpr int kCap = (1 << CELTY_RUN_BITS) - 1;   // largest run a padding entry carries
constexpr int kColBlock = 512;                      // columns per work item
constexpr int kChunk = 64;                          // groups per interleave chunk (a wavefront's lanes)
constexpr int32_t kMaxRows16 = 16376;               // tile rows of ROWS16: 4 * (R + 7) fits in 16 bits

inline bool stored(const uint16_t* W, int64_t ldw, const uint8_t* mask, int64_t ldm, int64_t r,
                   int64_t k) {
  if ((W[r * ldw + k] & 0x7FFFu) == 0) return false;   // +0 / -0 are never stored
  return mask == nullptr || mask[r * ldm + k] != 0;
}

// Exact value of an fp16 bit pattern (finite or not).
float half_bits_to_float(uint16_t h) {
  const uint32_t sign = uint32_t(h >> 15) << 31;
  const uint32_t exp = (h >> 10) & 0x1Fu, man = h & 0x3FFu;
  uint32_t bits;
  if (exp == 0x1F) {
    bits = sign | 0x7F800000u | (man << 13);
  } else if (exp != 0) {
    bits = sign | ((exp + 112u) << 23) | (man << 13);
  } else if (man == 0) {
    bits = sign;
  } else {   // subnormal: normalise
    int e = 113;
    uint32_t m = man;
    while ((m & 0x400u) == 0) {
      m <<= 1;
      --e;
    }
    bits = sign | (uint32_t(e) << 23) | ((m & 0x3FFu) << 13);
  }
  float f;
  std::memcpy(&f, &bits, sizeof f);
  return f;
}

struct Item {
  int32_t t, k0, k1;
};

std::vector<Item> make_items(int32_t T, int32_t K) {
  std::vector<Item> items;
  for (int32_t t = 0; t < T; ++t)
    for (int32_t k0 = 0; k0 < K; k0 += kColBlock) items.push_back({t, k0, std::min(K, k0 + kColBlock)});
  return items;
}

// Runs fn(item_index) over all items on n_threads workers.  Returns false if
// a worker could not be started or an item threw (its scratch could not be
// allocated); the caller maps this to ENOMEM.  No exception leaves a worker.
template <class Fn>
bool parallel_items(size_t n_items, int32_t n_threads, Fn fn) {
  unsigned hw = std::thread::hardware_concurrency();
  size_t nt = n_threads > 0 ? size_t(n_threads) : size_t(hw ? hw : 1);
  nt = std::max<size_t>(1, std::min(nt, n_items));
  std::atomic<size_t> next{0};
  std::atomic<bool> failed{false};
  auto worker = [&]() {
    for (size_t i = next.fetch_add(1); i < n_items; i = next.fetch_add(1)) {
      try {
        fn(i);
      } catch (...) {
        failed.store(true);
      }
    }
  };
  std::vector<std::thread> pool;
  try {
    for (size_t i = 1; i < nt; ++i) pool.emplace_back(worker);
  } catch (...) {
    for (auto& th : pool) th.join();
    return false;
  }
  worker();
  for (auto& th : pool) th.join();
  return !failed.load();
}

// Counts entries per segment of one item; writes groups per segment into
// seg_groups (indexed s - (t*K + k0)) when non-null and adds the totals.
void count_item(const uint16_t* W, int64_t ldw, const uint8_t* mask, int64_t ldm, int32_t M,
                int32_t R, bool bridge, const Item& it, std::vector<int32_t>& last, std::vector<int64_t>& cnt,
                int64_t& nnz, int64_t& pad, int64_t& groups, uint32_t* seg_groups) {
  const int32_t nk = it.k1 - it.k0;
  const int64_t r0 = int64_t(it.t) * R, r1 = std::min<int64_t>(M, r0 + R);
  std::fill(last.begin(), last.begin() + nk, -1);
  std::fill(cnt.begin(), cnt.begin() + nk, 0);
  for (int64_t r = r0; r < r1; ++r) {
    const int32_t rel = int32_t(r - r0);
    for (int32_t j = 0; j < nk; ++j) {
      if (!stored(W, ldw, mask, ldm, r, it.k0 + j)) continue;
      const int32_t np = bridge ? (rel - last[j] - 1) / (kCap + 1) : 0;   // padding entries before it
      cnt[j] += np + 1;
      pad += np;
      ++nnz;
      last[j] = rel;
    }
  }
  for (int32_t j = 0; j < nk; ++j) {
    const int64_t g = (cnt[j] + CELTY_GROUP - 1) / CELTY_GROUP;
    groups += g;
    if (seg_groups) seg_groups[j] = uint32_t(g);
  }
}

celty_status check_common(const uint16_t* W, int64_t ldw, const uint8_t* mask, int64_t ldm,
                          int32_t M, int32_t K, int32_t R, int32_t layout) {
  if (!W || M < 1 || K < 1 || R < 1 || ldw < K) return CELTY_EINVAL;
  if (mask && ldm < K) return CELTY_EINVAL;
  if (layout != CELTY_LAYOUT_RLC && layout != CELTY_LAYOUT_ROWS16 && layout != CELTY_LAYOUT_INTERLEAVED)
    return CELTY_EINVAL;
  if (layout == CELTY_LAYOUT_ROWS16 && R > kMaxRows16) return CELTY_EINVAL;
  return CELTY_OK;
}

// Lane-interleaved order of one segment's n groups (entries in row order in
// values[0 .. 8n) and the packed runs[0 .. n)): within each chunk of
// gc <= 64 groups, row-order entry e moves to group e % gc, slot e / gc
// (inverse = true moves it back).  tv and tr are scratch of 8 * 64 entries.
void interleave_segment(uint16_t* values, uint32_t* runs, int64_t n, bool inverse, uint16_t* tv, uint8_t* tr) {
  for (int64_t c0 = 0; c0 < n; c0 += kChunk) {
    const int64_t gc = std::min<int64_t>(kChunk, n - c0);
    uint16_t* v = values + c0 * CELTY_GROUP;
    uint32_t* r = runs + c0;
    for (int64_t e = 0; e < gc * CELTY_GROUP; ++e) {
      tv[e] = v[e];
      tr[e] = uint8_t((r[e / CELTY_GROUP] >> (4 * (e % CELTY_GROUP))) & 0xFu);
    }
    std::fill(r, r + gc, 0u);
    for (int64_t e = 0; e < gc * CELTY_GROUP; ++e) {
      const int64_t stored = (e % gc) * CELTY_GROUP + e / gc;   // group e % gc, slot e / gc
      const int64_t from = inverse ? stored : e, to = inverse ? e : stored;
      v[to] = tv[from];
      r[to / CELTY_GROUP] |= uint32_t(tr[from]) << (4 * (to % CELTY_GROUP));
    }
  }
}

}  // namespace

extern "C" celty_status celty_encode_plan(const uint16_t* W, int64_t ldw, const uint8_t* mask,
                                          int64_t ldm, int32_t M, int32_t K, int32_t R, int32_t layout,
                                          int64_t* n_groups, int64_t* n_nnz, int64_t* n_pad) {
  if (!n_groups || !n_nnz || !n_pad) return CELTY_EINVAL;
  if (celty_status st = check_common(W, ldw, mask, ldm, M, K, R, layout)) return st;
  try {
    const int32_t T = int32_t((int64_t(M) + R - 1) / R);
    const std::vector<Item> items = make_items(T, K);
    std::vector<int64_t> nnz(items.size()), pad(items.size()), grp(items.size());
    bool ok = parallel_items(items.size(), 0, [&](size_t i) {
      std::vector<int32_t> last(kColBlock);
      std::vector<int64_t> cnt(kColBlock);
      int64_t a = 0, b = 0, c = 0;
      count_item(W, ldw, mask, ldm, M, R, layout != CELTY_LAYOUT_ROWS16, items[i], last, cnt, a, b, c, nullptr);
      nnz[i] = a;
      pad[i] = b;
      grp[i] = c;
    });
    if (!ok) return CELTY_ENOMEM;
    int64_t A = 0, B = 0, C = 0;
    for (size_t i = 0; i < items.size(); ++i) {
      A += nnz[i];
      B += pad[i];
      C += grp[i];
    }
    if (C > int64_t(UINT32_MAX)) return CELTY_EOVERFLOW;
    *n_groups = C;
    *n_nnz = A;
    *n_pad = B;
    return CELTY_OK;
  } catch (const std::bad_alloc&) {
    return CELTY_ENOMEM;
  } catch (...) {
    return CELTY_ENOMEM;
  }
}

extern "C" celty_status celty_encode(const uint16_t* W, int64_t ldw, const uint8_t* mask,
                                     int64_t ldm, int32_t M, int32_t K, int32_t R, int32_t layout,
                                     uint32_t* gptr, uint16_t* values, uint32_t* runs, uint16_t* colmax,
                                     int64_t n_groups, celty_rlc_csc* out, int32_t n_threads) {
  if (celty_status st = check_common(W, ldw, mask, ldm, M, K, R, layout)) return st;
  if (!gptr || !out || !colmax || n_threads < 0 || n_groups < 0) return CELTY_EINVAL;
  if (n_groups > 0 && (!values || !runs)) return CELTY_EINVAL;
  const bool rows16 = layout == CELTY_LAYOUT_ROWS16;
  if ((reinterpret_cast<uintptr_t>(values) & 15u) || (reinterpret_cast<uintptr_t>(runs) & (rows16 ? 15u : 3u)) ||
      (reinterpret_cast<uintptr_t>(gptr) & 3u) || (reinterpret_cast<uintptr_t>(colmax) & 3u))
    return CELTY_EINVAL;
  if (n_groups > int64_t(UINT32_MAX)) return CELTY_EOVERFLOW;
  try {
    const int32_t T = int32_t((int64_t(M) + R - 1) / R);
    const int64_t nseg = int64_t(T) * K;
    const std::vector<Item> items = make_items(T, K);
    std::vector<int64_t> nnz(items.size()), pad(items.size());
    // largest |value| bits of column k within tile t, at t*K + k (each item
    // writes only its own columns of its own tile)
    std::vector<uint16_t> tile_colmax(size_t(nseg), 0);

    // pass 1: groups per segment, written into gptr[s] (then scanned in place)
    bool ok = parallel_items(items.size(), n_threads, [&](size_t i) {
      const Item& it = items[i];
      std::vector<int32_t> last(kColBlock);
      std::vector<int64_t> cnt(kColBlock);
      int64_t a = 0, b = 0, c = 0;
      count_item(W, ldw, mask, ldm, M, R, !rows16, it, last, cnt, a, b, c, gptr + int64_t(it.t) * K + it.k0);
      nnz[i] = a;
      pad[i] = b;
    });
    if (!ok) return CELTY_ENOMEM;
    int64_t acc = 0;
    for (int64_t s = 0; s < nseg; ++s) {
      const int64_t g = gptr[s];
      gptr[s] = uint32_t(acc);
      acc += g;
      if (acc > int64_t(UINT32_MAX)) return CELTY_EOVERFLOW;
    }
    if (acc != n_groups) return CELTY_EINVAL;
    gptr[nseg] = uint32_t(acc);

    // pass 2: fill.  Each item owns groups [gptr[t*K+k0], gptr[t*K+k1]).
    ok = parallel_items(items.size(), n_threads, [&](size_t i) {
      const Item& it = items[i];
      const int32_t nk = it.k1 - it.k0;
      const int64_t sbase = int64_t(it.t) * K + it.k0;
      const int64_t g0 = gptr[sbase], g1 = gptr[sbase + nk];
      const int64_t run_words = rows16 ? 4 : 1;   // words of row information per group
      std::memset(values + g0 * CELTY_GROUP, 0, size_t(g1 - g0) * CELTY_GROUP * sizeof(uint16_t));
      std::memset(runs + g0 * run_words, 0, size_t(g1 - g0) * run_words * sizeof(uint32_t));
      uint16_t* rows = reinterpret_cast<uint16_t*>(runs);   // ROWS16: entry e's offset at rows[e]
      std::vector<int32_t> last(nk, -1);
      std::vector<int64_t> pos(nk);   // next entry index (absolute) of each segment
      for (int32_t j = 0; j < nk; ++j) pos[j] = int64_t(gptr[sbase + j]) * CELTY_GROUP;
      auto emit = [&](int32_t j, uint16_t v, uint32_t run) {
        const int64_t e = pos[j]++;
        values[e] = v;
        runs[e / CELTY_GROUP] |= run << (4 * (e % CELTY_GROUP));
      };
      const int64_t r0 = int64_t(it.t) * R, r1 = std::min<int64_t>(M, r0 + R);
      for (int64_t r = r0; r < r1; ++r) {
        const int32_t rel = int32_t(r - r0);
        for (int32_t j = 0; j < nk; ++j) {
          if (!stored(W, ldw, mask, ldm, r, it.k0 + j)) continue;
          const uint16_t v = W[r * ldw + it.k0 + j];
          if (rows16) {
            const int64_t e = pos[j]++;
            values[e] = v;
            rows[e] = uint16_t(rel);
          } else {
            int32_t gap = rel - last[j] - 1;
            while (gap > kCap) {          // padding first, carrying the largest run
              emit(j, 0, uint32_t(kCap));
              gap -= kCap + 1;
            }
            emit(j, v, uint32_t(gap));
          }
          uint16_t& cm = tile_colmax[size_t(sbase + j)];
          cm = std::max<uint16_t>(cm, uint16_t(v & 0x7FFFu));   // magnitude bits order like the values
          last[j] = rel;
        }
      }
      // alignment entries: (0, 0) from the memset for runs; for row offsets,
      // value 0 at the segment's last stored row
      if (rows16) {
        for (int32_t j = 0; j < nk; ++j)
          for (int64_t e = pos[j]; e < int64_t(gptr[sbase + j + 1]) * CELTY_GROUP; ++e) rows[e] = uint16_t(last[j]);
      }
      if (layout == CELTY_LAYOUT_INTERLEAVED) {
        std::vector<uint16_t> tv(kChunk * CELTY_GROUP);
        std::vector<uint8_t> tr(kChunk * CELTY_GROUP);
        for (int32_t j = 0; j < nk; ++j) {
          const int64_t a = gptr[sbase + j], b = gptr[sbase + j + 1];
          interleave_segment(values + a * CELTY_GROUP, runs + a, b - a, false, tv.data(), tr.data());
        }
      }
    });
    if (!ok) return CELTY_ENOMEM;

    int64_t A = 0, B = 0;
    for (size_t i = 0; i < items.size(); ++i) {
      A += nnz[i];
      B += pad[i];
    }
    uint16_t mbits = 0;
    for (int32_t k = 0; k < K; ++k) {
      uint16_t m = 0;
      for (int32_t t = 0; t < T; ++t) m = std::max(m, tile_colmax[size_t(t) * K + k]);
      colmax[k] = m;
      mbits = std::max(mbits, m);
    }
    out->version = CELTY_FORMAT_VERSION;
    out->M = M;
    out->K = K;
    out->R = R;
    out->T = T;
    out->run_bits = CELTY_RUN_BITS;
    out->n_groups = n_groups;
    out->n_entries = A + B;
    out->n_nnz = A;
    out->n_pad = B;
    out->max_abs = half_bits_to_float(mbits);
    out->layout = layout;
    out->gptr = gptr;
    out->values = values;
    out->runs = runs;
    out->colmax = colmax;
    return CELTY_OK;
  } catch (...) {
    return CELTY_ENOMEM;
  }
}

namespace {

// Decodes the RLC entries of every segment (row order) into W_out/mask_out
// and the counts; EFORMAT on a malformed stream.
celty_status decode_rlc(const celty_rlc_csc* enc, const uint16_t* values, const uint32_t* runs, uint16_t* W_out,
                        uint8_t* mask_out, int64_t& nnz, int64_t& pad, std::vector<uint16_t>& cmax) {
  const int32_t M = enc->M, K = enc->K, R = enc->R;
  const int64_t nseg = int64_t(enc->T) * K;
  for (int64_t s = 0; s < nseg; ++s) {
    const int64_t t = s / K, k = s % K;
    const int64_t hi = std::min<int64_t>(M, (t + 1) * int64_t(R));
    int64_t row = t * int64_t(R) - 1;
    const int64_t e0 = int64_t(enc->gptr[s]) * CELTY_GROUP, e1 = int64_t(enc->gptr[s + 1]) * CELTY_GROUP;
    int64_t last_real = e0 - 1;
    for (int64_t e = e0; e < e1; ++e)
      if (values[e] & 0x7FFFu) last_real = e;
    for (int64_t e = e0; e < e1; ++e) {
      const uint32_t run = (runs[e / CELTY_GROUP] >> (4 * (e % CELTY_GROUP))) & 0xFu;
      const uint16_t v = values[e];
      row += int64_t(run) + 1;
      if (e > last_real) {            // alignment entries must be (0, 0)
        if (run != 0 || v != 0) return CELTY_EFORMAT;
        continue;
      }
      if (v & 0x7FFFu) {
        if (row >= hi) return CELTY_EFORMAT;
        W_out[row * K + k] = v;
        if (mask_out) mask_out[row * K + k] = 1;
        cmax[size_t(k)] = std::max<uint16_t>(cmax[size_t(k)], uint16_t(v & 0x7FFFu));
        ++nnz;
      } else {
        ++pad;
      }
    }
  }
  return CELTY_OK;
}

// Row offsets: stored values in strictly increasing rows inside the tile,
// then alignment entries (0, the last stored offset).
celty_status decode_rows16(const celty_rlc_csc* enc, uint16_t* W_out, uint8_t* mask_out, int64_t& nnz,
                           std::vector<uint16_t>& cmax) {
  const int32_t M = enc->M, K = enc->K, R = enc->R;
  const int64_t nseg = int64_t(enc->T) * K;
  const uint16_t* rows = reinterpret_cast<const uint16_t*>(enc->runs);
  for (int64_t s = 0; s < nseg; ++s) {
    const int64_t t = s / K, k = s % K;
    const int64_t hi = std::min<int64_t>(M, (t + 1) * int64_t(R)) - t * int64_t(R);
    const int64_t e0 = int64_t(enc->gptr[s]) * CELTY_GROUP, e1 = int64_t(enc->gptr[s + 1]) * CELTY_GROUP;
    int64_t prev = -1;
    bool tail = false;
    for (int64_t e = e0; e < e1; ++e) {
      const uint16_t v = enc->values[e];
      const int64_t r = rows[e];
      if (v & 0x7FFFu) {
        if (tail || r >= hi || r <= prev) return CELTY_EFORMAT;
        W_out[(t * int64_t(R) + r) * K + k] = v;
        if (mask_out) mask_out[(t * int64_t(R) + r) * K + k] = 1;
        cmax[size_t(k)] = std::max<uint16_t>(cmax[size_t(k)], uint16_t(v & 0x7FFFu));
        ++nnz;
        prev = r;
      } else {
        if (v != 0 || prev < 0 || r != prev) return CELTY_EFORMAT;
        tail = true;
      }
    }
  }
  return CELTY_OK;
}

}  // namespace

extern "C" celty_status celty_decode(const celty_rlc_csc* enc, uint16_t* W_out, uint8_t* mask_out) {
  if (!enc || !W_out) return CELTY_EINVAL;
  if (enc->version != CELTY_FORMAT_VERSION || enc->run_bits != CELTY_RUN_BITS) return CELTY_EINVAL;
  const int32_t layout = enc->layout;
  if (layout != CELTY_LAYOUT_RLC && layout != CELTY_LAYOUT_ROWS16 && layout != CELTY_LAYOUT_INTERLEAVED)
    return CELTY_EINVAL;
  const int32_t M = enc->M, K = enc->K, R = enc->R, T = enc->T;
  if (M < 1 || K < 1 || R < 1 || T != int32_t((int64_t(M) + R - 1) / R) || enc->n_groups < 0)
    return CELTY_EINVAL;
  if (layout == CELTY_LAYOUT_ROWS16 && R > kMaxRows16) return CELTY_EINVAL;
  if (!enc->gptr || !enc->colmax || (enc->n_groups > 0 && (!enc->values || !enc->runs))) return CELTY_EINVAL;
  const int64_t nseg = int64_t(T) * K;
  const uint32_t* gptr = enc->gptr;
  if (gptr[0] != 0 || int64_t(gptr[nseg]) != enc->n_groups) return CELTY_EFORMAT;
  for (int64_t s = 0; s < nseg; ++s)
    if (gptr[s + 1] < gptr[s]) return CELTY_EFORMAT;
  std::memset(W_out, 0, size_t(M) * K * sizeof(uint16_t));
  if (mask_out) std::memset(mask_out, 0, size_t(M) * K);
  int64_t nnz = 0, pad = 0;
  std::vector<uint16_t> cmax;
  std::vector<uint16_t> dv;   // an interleaved stream put back in row order
  std::vector<uint32_t> dr;
  try {
    cmax.assign(size_t(K), 0);
    if (layout == CELTY_LAYOUT_INTERLEAVED) {
      dv.assign(enc->values, enc->values + enc->n_groups * CELTY_GROUP);
      dr.assign(enc->runs, enc->runs + enc->n_groups);
    }
  } catch (...) {
    return CELTY_ENOMEM;
  }
  celty_status st;
  if (layout == CELTY_LAYOUT_ROWS16) {
    st = decode_rows16(enc, W_out, mask_out, nnz, cmax);
  } else if (layout == CELTY_LAYOUT_INTERLEAVED) {
    uint16_t tv[kChunk * CELTY_GROUP];
    uint8_t tr[kChunk * CELTY_GROUP];
    for (int64_t s = 0; s < nseg; ++s)
      interleave_segment(dv.data() + int64_t(gptr[s]) * CELTY_GROUP, dr.data() + gptr[s], gptr[s + 1] - gptr[s],
                         true, tv, tr);
    st = decode_rlc(enc, dv.data(), dr.data(), W_out, mask_out, nnz, pad, cmax);
  } else {
    st = decode_rlc(enc, enc->values, enc->runs, W_out, mask_out, nnz, pad, cmax);
  }
  if (st != CELTY_OK) return st;
  if (nnz != enc->n_nnz || pad != enc->n_pad || nnz + pad != enc->n_entries) return CELTY_EFORMAT;
  uint16_t mbits = 0;
  for (int32_t k = 0; k < K; ++k) {
    if (enc->colmax[k] != cmax[size_t(k)]) return CELTY_EFORMAT;
    mbits = std::max(mbits, cmax[size_t(k)]);
  }
  if (enc->max_abs != half_bits_to_float(mbits)) return CELTY_EFORMAT;
  return CELTY_OK;
}
