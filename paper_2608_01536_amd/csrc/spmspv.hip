// Dual-sparse SpMSpV kernels for gfx950 (CDNA4) and their C ABI entry points.
//
// One launch computes y = W x_A (Sections 3.1-3.3):
//   * grid = (row tile t) x (slice c of x).  A workgroup selects the active
//     columns of its slice (|x_k| > tau; one block-wide scan of per-lane
//     counts: Section 3.1's column skip turned into stream compaction) and
//     drops columns whose segment in tile t is empty;
//   * the workgroup's compressed groups (8 entries = 16 B of fp16 values +
//     4 B of packed 4-bit runs) form one flat sequence, cut at group
//     boundaries into one contiguous range per wavefront (a segment may be
//     shared; a range that starts inside one first sums the runs of its
//     earlier groups to find its starting row; 16 wavefronts get shares
//     weighted by their rank on the SIMD);
//   * a wavefront walks its range 64*G groups per pass, keeping a ring of
//     passes in flight: each lane loads its groups with 128-bit and 32-bit
//     buffer loads (Section 3.1), turns the 8 runs of a group into 8
//     inclusive prefixes with byte-packed arithmetic, and combines lanes with
//     a wavefront scan that restarts at segment heads (Algorithm 1: prefix of
//     runs plus ordinal gives the row);
//   * each product value * x_k is exact in fp32 (two fp16 factors) and is
//     added into an LDS tile of the R output rows (Section 3.3's
//     scatter-accumulation in on-chip memory).  The tile holds int32 fixed
//     point on a per-workgroup grid 2^-s derived from the slice's own data:
//     B = n * max over its n kept columns of colmax[k] * |x_k| bounds every
//     row's sum of |products|, and 2^s puts B just below 2^30, so no row can
//     overflow (on gfx950 an LDS integer atomic add costs a small fraction of
//     an fp32 one);
//   * the slices of a row tile are merged with one returning 64-bit atomic
//     per row and slice on a fixed grid of 2^-33 (each slice's partial
//     clamped to +-4096, far above the partials of LLM layers) plus an
//     arrival count; a slice whose partial exceeds the clamp first adds the
//     excess to a second word on a grid of 2^-8 and flags it in the first,
//     so that the last slice also reads that word.  The slice that arrives
//     last writes y[row] in fp16 and clears the words for the next call.
//     With a single slice the tile goes straight to y.
//
// Variants of the same product (for the ablations of Sections 4.1-4.2; the
// default above is the paper's format in its stored order): 16-bit row
// offsets loaded instead of reconstructed, the runs in lane-interleaved order
// (each pass then holds whole chunks, and the eight slot prefixes come from
// packed wavefront scans), and an XOR-swizzled slot order of the LDS tile.
// Each forms the same products on the same grids, so its y is the default's
// bit for bit.

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <mutex>
#include <type_traits>

#include "celty.h"
#include "common.h"

namespace {

constexpr int kMaxLds = 160 * 1024;   // LDS per workgroup on gfx950
constexpr int kSlack = 8 + 128;       // tile rows past R: alignment entries, and the cap's reach
constexpr int kMaxSlices = 63;        // column slices per row tile (6-bit arrival count of the merge)
constexpr int kMaxCols = 8;           // columns per thread in the selection
// The merge's 64-bit ticket: a slice's clamped partial on the grid 2^-33
// plus a bias of kFineClamp (= 4096 on that grid) in bits 0..51, the count
// of clamped slices in bits 52..57 and the arrival count in bits 58..63.
constexpr long long kFineClamp = 1ll << 45;
constexpr unsigned long long kTicketExcess = 1ull << 52;
constexpr unsigned long long kTicketCount = 1ull << 58;
// Cache policy of the value loads: non-temporal (the nt bit of gfx950's
// buffer loads), so the streamed weights do not displace cached lines.
constexpr int kStreamPolicy = 2;

// Kernel variants: the row encodings of the format (layout field) and the
// LDS tile's slot order.
constexpr int kVarRlc = 0;           // 4-bit runs, plain tile
constexpr int kVarSwizzle = 1;       // 4-bit runs, tile row r at slot r ^ ((r >> 6) & 63)
constexpr int kVarRows16 = 2;        // 16-bit row offsets
constexpr int kVarInterleaved = 3;   // 4-bit runs in lane-interleaved order within chunks of 64 groups
constexpr int kChunk = 64;           // groups per interleave chunk

// Dynamic LDS of a workgroup (byte offsets; the int32 tile is at 0): the
// tile of R rows plus 7 alignment rows and 128 rows of slack that bound where
// a corrupt stream could write (a group base is capped at R + 7 and a group
// adds at most 128), rounded up to 64 rows so that the swizzled slot order
// (a permutation within aligned blocks of 64 rows) stays inside it; the
// selection's list of Kc segments; the walk's scratch (64 * scr_words ints
// per wavefront); the block scan's per-wavefront totals (3 words each).  The
// host sizes the launch with the same function.
struct LdsLayout {
  int tile_slots, seg_off, scr_off, misc_off, bytes;
};
__host__ __device__ constexpr int align16(int v) { return (v + 15) & ~15; }
__host__ __device__ constexpr int tile_slots_of(int R) { return (R + kSlack + 63) & ~63; }
__host__ __device__ constexpr LdsLayout lds_layout(int R, int Kc, int waves, int scr_words) {
  return LdsLayout{tile_slots_of(R), 4 * tile_slots_of(R), 4 * tile_slots_of(R) + 16 * Kc,
                   4 * tile_slots_of(R) + 16 * Kc + 256 * waves * scr_words,
                   align16(4 * tile_slots_of(R) + 16 * Kc + 256 * waves * scr_words + 12 * waves)};
}
// Scratch ints per lane of the walk: one per group of a pass, four for the
// interleaved layout's packed per-slot scans.
__host__ __device__ constexpr int scr_words_of(int groups, int var) { return var == kVarInterleaved ? 4 : groups; }

// Tile slot of row r (as a byte offset, 4 * r) in the swizzled order:
// r ^ ((r >> 6) & 63), a permutation within each aligned block of 64 rows.
__device__ __forceinline__ uint32_t swizzle4(uint32_t a) { return a ^ ((a >> 6) & 0xFCu); }

struct SegInfo {
  uint32_t gstart;   // first group of the segment in the values/runs arrays
  uint32_t off;      // first group of the segment in the workgroup's flat sequence
  uint32_t cnt;      // groups in the segment (> 0)
  float xs;          // x_k * 2^s (s: the workgroup's fixed-point scale)
};

__device__ __forceinline__ unsigned short float_to_half_bits(float v) {
  return __half_as_ushort(__float2half_rn(v));
}

// Orders LDS writes of some lanes before LDS reads of other lanes of the
// same wavefront.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The same pattern with max: lane 63 ends with the wavefront maximum.
__device__ __forceinline__ uint32_t wave_inclusive_max(uint32_t v) {
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x111, 0xF, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x112, 0xF, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x114, 0xF, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x118, 0xF, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x142, 0xA, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x143, 0xC, 0xF, false)));
  return v;
}

// Inclusive scan over the 16 lanes of each DPP row.
__device__ __forceinline__ uint32_t row_inclusive_scan(uint32_t v) {
  v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x111, 0xF, 0xF, false));
  v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x112, 0xF, 0xF, false));
  v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x114, 0xF, 0xF, false));
  v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x118, 0xF, 0xF, false));
  return v;
}
__device__ __forceinline__ uint32_t row_inclusive_max(uint32_t v) {
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x111, 0xF, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x112, 0xF, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x114, 0xF, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x118, 0xF, 0xF, false)));
  return v;
}

// Block-wide: exclusive scans of a and b, their totals, and the maximum of m
// (WAVES <= 16).  Each wavefront's totals go to part[] (3*WAVES words, used
// once per launch); after the barrier lane l < WAVES of every wavefront reads
// wavefront l's totals and one row scan gives the offsets of all wavefronts.
template <int WAVES>
__device__ __forceinline__ void block_scan_select(uint32_t a, uint32_t b, uint32_t m, uint32_t& ea, uint32_t& eb,
                                                  uint32_t& ta, uint32_t& tb, uint32_t& tm, uint32_t* part) {
  static_assert(WAVES <= 16, "one DPP row holds the per-wavefront totals");
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const uint32_t ia = static_cast<uint32_t>(wave_inclusive_scan(static_cast<int>(a)));
  const uint32_t ib = static_cast<uint32_t>(wave_inclusive_scan(static_cast<int>(b)));
  const uint32_t im = wave_inclusive_max(m);
  if (lane == kWave - 1) {
    part[wv] = ia;
    part[WAVES + wv] = ib;
    part[2 * WAVES + wv] = im;
  }
  __syncthreads();
  uint32_t pa = 0, pb = 0, pm = 0;
  if (lane < WAVES) {
    pa = part[lane];
    pb = part[WAVES + lane];
    pm = part[2 * WAVES + lane];
  }
  const uint32_t sa = row_inclusive_scan(pa), sb = row_inclusive_scan(pb), sm = row_inclusive_max(pm);
  ta = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(sa), WAVES - 1));
  tb = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(sb), WAVES - 1));
  tm = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(sm), WAVES - 1));
  const uint32_t oa = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(sa - pa), wv));
  const uint32_t ob = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(sb - pb), wv));
  ea = oa + ia - a;
  eb = ob + ib - b;
}

// The grid 2^-s whose scale puts a bound b just below 2^top: with
// 2^(e-1) <= b < 2^e, s = top - e (clamped to [-64, 64]; 0 for b = 0; the
// exponent of a non-finite b reads as 0).
__device__ __forceinline__ int grid_scale(float b, int top) {
  if (!(b > 0.f)) return 0;
  return min(max(top - __builtin_amdgcn_frexp_expf(b), -64), 64);
}

// Start of wavefront w's range of the slice's n_grp groups.  A SIMD holds
// wavefronts w, w + 4, ... and over a long walk serves its later ones more
// slowly (with equal ranges, ranks w / 4 = 0..3 of 16 took 0.89, 0.94, 1.03
// and 1.14 times the mean walk at 28672 x 8192), so with 16 wavefronts the
// ranks get shares in proportion 80 : 72 : 56 : 48 (the best of a measured
// series; the speeds shift as the shares do), in units of n_grp / 1024:
// rank r's weight is byte r of 0x30384850 and the weight of the ranks
// below it is 16-bit field r of 0x340026001400000.  32-bit arithmetic (n_grp =
// 1024 q + m, n_grp < 2^27); otherwise equal shares (w * n_grp < 2^31).
template <int WAVES>
__device__ __forceinline__ uint32_t cut_of(int w, uint32_t n_grp) {
  if constexpr (WAVES == 16) {
    const uint32_t r = static_cast<uint32_t>(w) >> 2, m = static_cast<uint32_t>(w) & 3u;
    const uint32_t wt = (0x30384850u >> (8u * (r & 3u))) & 255u;
    const uint32_t below = r >= 4u ? 1024u : static_cast<uint32_t>(0x340026001400000ull >> (16u * r)) & 65535u;
    const uint32_t cum = below + m * wt;
    return (n_grp >> 10) * cum + (((n_grp & 1023u) * cum) >> 10);
  } else {
    return static_cast<uint32_t>(w) * n_grp / WAVES;
  }
}

// 4 * sum of (run + 1) over the 8 entries of a group (runs word rw).
__device__ __forceinline__ int group_span4(uint32_t rw) {
  return static_cast<int>(__builtin_amdgcn_sad_u8(((rw << 2) & 0x3C3C3C3Cu) + ((rw >> 2) & 0x3C3C3C3Cu), 0u, 32u));
}

// The segment that holds flat group `at` (at < the slice's group count), for
// a whole wavefront: the n_seg <= 64 * 64 segments, sorted by offset, are
// searched with two ballots, over every stride-th segment and then over the
// one bucket of stride segments that holds `at`.  Returns the segment's index
// and its gstart, off and cnt (wavefront-uniform; xs is left 0).
__device__ __forceinline__ int holding_segment(const SegInfo* seg, int n_seg, uint32_t at, int lane, SegInfo& r) {
  const int stride = (n_seg + kWave - 1) / kWave;   // <= 64
  const int s1 = min(lane * stride, n_seg - 1);
  const int c1 = __popcll(__ballot(seg[s1].off <= at));   // >= 1: segment 0 starts at 0
  const int lo = min((c1 - 1) * stride, n_seg - 1);
  const int hi = min(c1 * stride, n_seg);
  const SegInfo sg = seg[min(lo + lane, n_seg - 1)];
  const int c2 = __popcll(__ballot(lo + lane < hi && sg.off <= at));   // >= 1
  r.gstart = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(sg.gstart), c2 - 1));
  r.off = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(sg.off), c2 - 1));
  r.cnt = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(sg.cnt), c2 - 1));
  r.xs = 0.f;
  return lo + c2 - 1;
}

// fp16 (low or high half of a word) times an fp32 value, in one mixed-precision
// FMA; exact for the products formed here (11-bit by 11-bit significands).
__device__ __forceinline__ float mul_lo_f16(uint32_t w, float x) {
  float r;
  asm("v_fma_mix_f32 %0, %1, %2, 0 op_sel_hi:[1,0,0]" : "=v"(r) : "v"(w), "v"(x));
  return r;
}
__device__ __forceinline__ float mul_hi_f16(uint32_t w, float x) {
  float r;
  asm("v_fma_mix_f32 %0, %1, %2, 0 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(r) : "v"(w), "v"(x));
  return r;
}

// floor(v + 0.5) as int32 (v is within +-2^30 by the choice of scale).
__device__ __forceinline__ int round_to_fixed(float v) {
  int r;
  asm("v_cvt_rpi_i32_f32 %0, %1" : "=v"(r) : "v"(v));
  return r;
}

// Buffer resources for the values and runs arrays: 32-bit offsets, and the
// hardware returns zeros for any read past num_records, so a corrupt
// group-pointer array cannot read outside the arrays.
struct Streams {
  __amdgpu_buffer_rsrc_t values;
  __amdgpu_buffer_rsrc_t runs;
};

__device__ __forceinline__ Streams make_streams(const uint4* values, const uint32_t* runs, uint32_t n_groups,
                                                uint32_t run_bytes) {
  Streams st;
  st.values = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint4*>(values), static_cast<short>(0),
                                                static_cast<int>(n_groups * 16u), 0x00020000);
  st.runs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(runs), static_cast<short>(0),
                                              static_cast<int>(n_groups * run_bytes), 0x00020000);
  return st;
}

// One pass's input for a lane: G consecutive groups of the workgroup's flat
// sequence (8 entries each) and, per group, its segment's head and x.
template <int G>
struct Pass {
  uint4 v[G];        // 8 fp16 values per group
  uint32_t rw[G];    // 8 packed 4-bit runs per group
  uint4 rr[G];       // 8 16-bit row offsets per group (16-bit row layout)
  int hpos[G];       // flat position of the group's segment head relative to the pass start (< 0: earlier)
  float xs[G];       // scaled x_k of the group's column
  uint32_t live;     // bit i: group i holds data
  int sid63;         // segment of lane 63's last group (wavefront-uniform)
  uint32_t end63;    // its flat end (wavefront-uniform)
};

// Assigns the 64*G groups starting at flat position pb to lanes (lane l takes
// groups pb + G*l .. pb + G*l + G-1) and issues their loads.  icur is the
// segment holding group pb.  A pass at or past the end (pb >= pe) skips the
// assignment and has every lane idle.  scr holds 64*G ints per wavefront:
// segment heads are tagged with a negative value unique to the pass (the
// accumulation step stores non-negative prefix sums in the same array).
template <int G, bool ROWS16>
__device__ __forceinline__ void fetch_pass(Pass<G>& a, const Streams& st, const SegInfo* seg, int* scr,
                                           uint32_t pb, int icur, int i_end, uint32_t pe, int lane) {
  constexpr uint32_t P = kWave * G;
  a.live = 0u;
  a.sid63 = icur;
  a.end63 = pe;
  uint32_t gl[G];
#pragma unroll
  for (int i = 0; i < G; ++i) {
    a.hpos[i] = 0;
    a.xs[i] = 0.f;
    gl[i] = 0u;
  }
  if (pb < pe) {   // wavefront-uniform
    const int tag = -static_cast<int>(pb) - 1;
    // segments icur+1 .. icur+64G are the only ones that can start in the pass
#pragma unroll
    for (int m = 0; m < G; ++m) {
      const int j = icur + 1 + lane + kWave * m;
      if (j < i_end) {
        const uint32_t o = seg[j].off;
        if (o < pb + P) scr[o - pb] = tag;
      }
    }
    wave_lds_sync();
    uint32_t fl = 0u;   // bit i: position G*lane + i is a segment head
#pragma unroll
    for (int i = 0; i < G; ++i) fl |= (scr[G * lane + i] == tag ? 1u : 0u) << i;
    const uint32_t nh = __popc(fl);
    // heads in the positions of the lanes below, from the bits of nh
    int cum = 0;
#pragma unroll
    for (int b = 0; (1 << b) <= G; ++b) cum += static_cast<int>(lanes_below(__ballot((nh >> b) & 1u))) << b;
    int sid = icur;
    uint32_t end = pe;
#pragma unroll
    for (int i = 0; i < G; ++i) {
      cum += (fl >> i) & 1u;
      sid = min(icur + cum, i_end - 1);
      const SegInfo si = seg[sid];
      const uint32_t f = pb + static_cast<uint32_t>(G * lane + i);
      const bool lv = f < pe;
      a.hpos[i] = static_cast<int>(si.off) - static_cast<int>(pb);
      a.xs[i] = si.xs;
      gl[i] = lv ? si.gstart + (f - si.off) : 0u;
      a.live |= (lv ? 1u : 0u) << i;
      end = si.off + si.cnt;
    }
    a.sid63 = __builtin_amdgcn_readlane(sid, kWave - 1);
    a.end63 = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(end), kWave - 1));
  }
  // Loads are issued by every lane of every pass (idle lanes and idle passes
  // read group 0 and drop it), so the wait for one pass's data can leave the
  // later passes' loads in flight.  The values are streamed non-temporally
  // (each of their lines is read once); the runs keep the default policy,
  // since a pass's 256 bytes of runs usually share a line with the next pass.
#pragma unroll
  for (int i = 0; i < G; ++i) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(st.values, static_cast<int>(gl[i] << 4), 0, kStreamPolicy);
    a.v[i] = make_uint4(v[0], v[1], v[2], v[3]);
    if constexpr (ROWS16) {
      const auto r = __builtin_amdgcn_raw_buffer_load_b128(st.runs, static_cast<int>(gl[i] << 4), 0, kStreamPolicy);
      a.rr[i] = make_uint4(r[0], r[1], r[2], r[3]);
    } else {
      a.rw[i] = __builtin_amdgcn_raw_buffer_load_b32(st.runs, static_cast<int>(gl[i] << 2), 0, 0);
    }
  }
}

// The segment holding the first group of the pass after the one fetched at
// flat position pb (wavefront-uniform).
template <int G>
__device__ __forceinline__ int next_pass_segment(const Pass<G>& a, uint32_t pb, int i_end) {
  return min(a.end63 > pb + kWave * G ? a.sid63 : a.sid63 + 1, i_end - 1);
}

// a + byte Q of b in one VALU operation (SDWA source select).
template <int Q>
__device__ __forceinline__ uint32_t add_byte(uint32_t a, uint32_t b) {
  uint32_t r;
  if constexpr (Q == 0)
    asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
        : "=v"(r) : "v"(a), "v"(b));
  else if constexpr (Q == 1)
    asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
        : "=v"(r) : "v"(a), "v"(b));
  else if constexpr (Q == 2)
    asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2"
        : "=v"(r) : "v"(a), "v"(b));
  else
    asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
        : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Adds entry j's product at LDS byte address a + 4 * (j + 1), the constant in
// the instruction's offset field.  (LDS operations complete in order, so the
// compiler's waits for its own LDS accesses stay correct around this one; the
// clobber keeps it in order with them.)
template <int J>
__device__ __forceinline__ void tile_add(uint32_t a, int v) {
  asm volatile("ds_add_u32 %0, %1 offset:%2" : : "v"(a), "v"(v), "i"(4 * (J + 1)) : "memory");
}
// The same at LDS byte address a exactly.
__device__ __forceinline__ void tile_add_at(uint32_t a, int v) {
  asm volatile("ds_add_u32 %0, %1" : : "v"(a), "v"(v) : "memory");
}

// a + the 16-bit half Q of b in one VALU operation (SDWA source select).
template <int Q>
__device__ __forceinline__ uint32_t add_word(uint32_t a, uint32_t b) {
  uint32_t r;
  if constexpr (Q == 0)
    asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:WORD_0"
        : "=v"(r) : "v"(a), "v"(b));
  else
    asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:WORD_1"
        : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Both 16-bit halves of w, each clamped to the halves of c.
__device__ __forceinline__ uint32_t min_u16x2(uint32_t w, uint32_t c) {
  uint32_t r;
  asm("v_pk_min_u16 %0, %1, %2" : "=v"(r) : "v"(w), "v"(c));
  return r;
}

// Decodes one pass and adds its products into the fixed-point tile at LDS
// byte address tile_lds.  Row arithmetic is done on byte offsets, 4 * row: a
// group's runs r_0..r_7 put entry j at 4 * (base + sum_{i<=j} (r_i + 1)), so
// one running address advances by the byte 4 * r_j per entry and the
// constant 4 * (j + 1) is an immediate.  Returns the
// segment-relative sum of 4 * (run + 1) through lane 63's last group (the
// carry when that segment goes on into the next pass), wavefront-uniform.
template <int G, bool SWZ>
__device__ __forceinline__ int accumulate_pass(const Pass<G>& a, int carry4, int base4_cap, uint32_t tile_lds,
                                               int* scr, int lane) {
  uint32_t R4e[G], R4o[G];
  int S4[G], C4[G];
  int T = 0;
#pragma unroll
  for (int i = 0; i < G; ++i) {
    const bool lv = (a.live >> i) & 1u;
    const uint32_t rw = lv ? a.rw[i] : 0u;
    R4e[i] = (rw << 2) & 0x3C3C3C3Cu;   // byte k: 4 * r_{2k}
    R4o[i] = (rw >> 2) & 0x3C3C3C3Cu;   // byte k: 4 * r_{2k+1}
    // 4 * sum of (run + 1) over the group
    S4[i] = lv ? static_cast<int>(__builtin_amdgcn_sad_u8(R4e[i] + R4o[i], 0u, 32u)) : 0;
    C4[i] = T;   // before the group, within the lane
    T += S4[i];
  }
  const int incl = wave_inclusive_scan(T);
  const int X = incl - T;   // before the lane's first group, within the pass
  // prefix before every flat position of the pass, for the segment heads
#pragma unroll
  for (int i = 0; i < G; ++i) scr[G * lane + i] = X + C4[i];
  wave_lds_sync();
  int tail = 0;
#pragma unroll
  for (int i = 0; i < G; ++i) {
    const int Y = X + C4[i];
    const int at_head = scr[max(a.hpos[i], 0)];
    const int rel4 = a.hpos[i] >= 0 ? Y - at_head : Y + carry4;   // segment-relative
    // entry j lands at base4 + sum_{i<=j} 4 r_i + 4 (j + 1) with base4 >= -4;
    // the cap keeps even a corrupt stream inside the tile's slack
    const uint32_t base4 = static_cast<uint32_t>(min(rel4 - 4, base4_cap)) + (SWZ ? 0u : tile_lds);
    if constexpr (SWZ) {
      if ((a.live >> i) & 1u) {
        // the running offset is tile-relative and advances by 4 (r_j + 1)
        // (each byte at most 64, so adding 4 per byte cannot carry); the
        // slot order is applied to it, then the tile's address added
        const float xs = a.xs[i];
        const uint32_t E = R4e[i] + 0x04040404u, O = R4o[i] + 0x04040404u;
        uint32_t ad = base4;
        ad = add_byte<0>(ad, E);
        tile_add_at(swizzle4(ad) + tile_lds, round_to_fixed(mul_lo_f16(a.v[i].x, xs)));
        ad = add_byte<0>(ad, O);
        tile_add_at(swizzle4(ad) + tile_lds, round_to_fixed(mul_hi_f16(a.v[i].x, xs)));
        ad = add_byte<1>(ad, E);
        tile_add_at(swizzle4(ad) + tile_lds, round_to_fixed(mul_lo_f16(a.v[i].y, xs)));
        ad = add_byte<1>(ad, O);
        tile_add_at(swizzle4(ad) + tile_lds, round_to_fixed(mul_hi_f16(a.v[i].y, xs)));
        ad = add_byte<2>(ad, E);
        tile_add_at(swizzle4(ad) + tile_lds, round_to_fixed(mul_lo_f16(a.v[i].z, xs)));
        ad = add_byte<2>(ad, O);
        tile_add_at(swizzle4(ad) + tile_lds, round_to_fixed(mul_hi_f16(a.v[i].z, xs)));
        ad = add_byte<3>(ad, E);
        tile_add_at(swizzle4(ad) + tile_lds, round_to_fixed(mul_lo_f16(a.v[i].w, xs)));
        ad = add_byte<3>(ad, O);
        tile_add_at(swizzle4(ad) + tile_lds, round_to_fixed(mul_hi_f16(a.v[i].w, xs)));
      }
    } else if ((a.live >> i) & 1u) {
      const float xs = a.xs[i];
      uint32_t ad = base4;
      ad = add_byte<0>(ad, R4e[i]);
      tile_add<0>(ad, round_to_fixed(mul_lo_f16(a.v[i].x, xs)));
      ad = add_byte<0>(ad, R4o[i]);
      tile_add<1>(ad, round_to_fixed(mul_hi_f16(a.v[i].x, xs)));
      ad = add_byte<1>(ad, R4e[i]);
      tile_add<2>(ad, round_to_fixed(mul_lo_f16(a.v[i].y, xs)));
      ad = add_byte<1>(ad, R4o[i]);
      tile_add<3>(ad, round_to_fixed(mul_hi_f16(a.v[i].y, xs)));
      ad = add_byte<2>(ad, R4e[i]);
      tile_add<4>(ad, round_to_fixed(mul_lo_f16(a.v[i].z, xs)));
      ad = add_byte<2>(ad, R4o[i]);
      tile_add<5>(ad, round_to_fixed(mul_hi_f16(a.v[i].z, xs)));
      ad = add_byte<3>(ad, R4e[i]);
      tile_add<6>(ad, round_to_fixed(mul_lo_f16(a.v[i].w, xs)));
      ad = add_byte<3>(ad, R4o[i]);
      tile_add<7>(ad, round_to_fixed(mul_hi_f16(a.v[i].w, xs)));
    }
    if (i == G - 1) tail = rel4 + S4[i];
  }
  return __builtin_amdgcn_readlane(tail, kWave - 1);
}

// 16-bit row layout: each entry's row offset is loaded, so there is nothing
// to reconstruct.  Offsets are clamped to R + 7 (the tile's slack), four
// times each (4 * (R + 7) < 2^16), and added to the tile's address per entry.
template <int G>
__device__ __forceinline__ void accumulate_pass_rows16(const Pass<G>& a, uint32_t cap_rows2, uint32_t tile_lds) {
#pragma unroll
  for (int i = 0; i < G; ++i) {
    if ((a.live >> i) & 1u) {
      const float xs = a.xs[i];
      const uint32_t r0 = min_u16x2(a.rr[i].x, cap_rows2) << 2, r1 = min_u16x2(a.rr[i].y, cap_rows2) << 2;
      const uint32_t r2 = min_u16x2(a.rr[i].z, cap_rows2) << 2, r3 = min_u16x2(a.rr[i].w, cap_rows2) << 2;
      tile_add_at(add_word<0>(tile_lds, r0), round_to_fixed(mul_lo_f16(a.v[i].x, xs)));
      tile_add_at(add_word<1>(tile_lds, r0), round_to_fixed(mul_hi_f16(a.v[i].x, xs)));
      tile_add_at(add_word<0>(tile_lds, r1), round_to_fixed(mul_lo_f16(a.v[i].y, xs)));
      tile_add_at(add_word<1>(tile_lds, r1), round_to_fixed(mul_hi_f16(a.v[i].y, xs)));
      tile_add_at(add_word<0>(tile_lds, r2), round_to_fixed(mul_lo_f16(a.v[i].z, xs)));
      tile_add_at(add_word<1>(tile_lds, r2), round_to_fixed(mul_hi_f16(a.v[i].z, xs)));
      tile_add_at(add_word<0>(tile_lds, r3), round_to_fixed(mul_lo_f16(a.v[i].w, xs)));
      tile_add_at(add_word<1>(tile_lds, r3), round_to_fixed(mul_hi_f16(a.v[i].w, xs)));
    }
  }
}

// ---- interleaved layout ---------------------------------------------------
// A pass holds whole chunks only: a chunk's eight slots are consecutive runs
// of the row order across its lanes, so decoding slot j needs the runs of
// every lane of the chunk.  The wavefront's range and its passes are cut at
// chunk boundaries: at a segment's head and every 64 groups after it, and
// at its end.

// The first chunk boundary at or after flat group `at` (wavefront-uniform).
__device__ __forceinline__ uint32_t chunk_boundary(const SegInfo* seg, int n_seg, uint32_t n_grp, uint32_t at,
                                                   int lane) {
  if (at >= n_grp) return n_grp;
  SegInfo s;
  holding_segment(seg, n_seg, at, lane, s);
  const uint32_t b = s.off + ((at - s.off + static_cast<uint32_t>(kChunk - 1)) & ~static_cast<uint32_t>(kChunk - 1));
  return min(b, s.off + s.cnt);
}

struct PassIl {
  uint4 v;           // 8 fp16 values (slots 0..7)
  uint32_t rw;       // their 8 packed 4-bit runs
  float xs;          // scaled x_k of the group's column
  int hl, el;        // lanes of the group's chunk head and last group, within the pass
  bool first;        // the chunk is its segment's first (else it goes on from the previous pass, at lane 0)
  bool live;
  uint32_t pend;     // flat end of the pass (wavefront-uniform)
  int next_seg;      // segment holding pend (wavefront-uniform)
  bool cont;         // the segment of the pass's last chunk goes on past pend (wavefront-uniform)
};

// Assigns the chunks that fit whole in [pb, min(pb + 64, pe)) to lanes (lane
// l takes group pb + l) and issues their loads; pb is a chunk boundary.  An
// idle pass (pb >= pe) has every lane inactive and pend = pb.
__device__ __forceinline__ void fetch_pass_il(PassIl& a, const Streams& st, const SegInfo* seg, int* scr,
                                              uint32_t pb, int icur, int i_end, uint32_t pe, int lane) {
  a.live = false;
  a.xs = 0.f;
  a.hl = a.el = 0;
  a.first = true;
  a.pend = pb;
  a.next_seg = icur;
  a.cont = false;
  uint32_t gl = 0u;
  if (pb < pe) {   // wavefront-uniform
    const int tag = -static_cast<int>(pb) - 1;
    const int j = icur + 1 + lane;   // only segments icur+1 .. icur+64 can start in the pass
    if (j < i_end) {
      const uint32_t o = seg[j].off;
      if (o < pb + kWave) scr[o - pb] = tag;
    }
    wave_lds_sync();
    const uint32_t fl = scr[lane] == tag ? 1u : 0u;
    const int cum = static_cast<int>(lanes_below(__ballot(fl))) + static_cast<int>(fl);
    const int sid = min(icur + cum, i_end - 1);
    const SegInfo si = seg[sid];
    const uint32_t f = pb + static_cast<uint32_t>(lane);
    const uint32_t fe = min(pb + static_cast<uint32_t>(kWave), pe);
    const int ll = static_cast<int>(fe - 1u - pb);   // the last lane that may hold a group
    const uint32_t s_off = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(si.off), ll));
    const uint32_t s_end = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(si.off + si.cnt), ll));
    const int s_id = __builtin_amdgcn_readlane(sid, ll);
    // the last chunk boundary at or before fe
    const uint32_t pend = s_end > fe ? s_off + ((fe - s_off) & ~static_cast<uint32_t>(kChunk - 1)) : fe;
    a.pend = pend;
    a.next_seg = min(pend < s_end ? s_id : s_id + 1, i_end - 1);
    a.cont = s_end > pend;
    const bool lv = f < pend;
    const uint32_t h = si.off + ((f - si.off) & ~static_cast<uint32_t>(kChunk - 1));
    const uint32_t ce = min(h + static_cast<uint32_t>(kChunk), si.off + si.cnt);
    a.hl = static_cast<int>(h - pb);
    a.el = static_cast<int>(ce - 1u - pb);
    a.first = h == si.off;
    a.xs = si.xs;
    a.live = lv;
    gl = lv ? si.gstart + (f - si.off) : 0u;
  }
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(st.values, static_cast<int>(gl << 4), 0, kStreamPolicy);
  a.v = make_uint4(v[0], v[1], v[2], v[3]);
  a.rw = __builtin_amdgcn_raw_buffer_load_b32(st.runs, static_cast<int>(gl << 2), 0, 0);
}

// Decodes one interleaved pass and adds its products.  Slot j of the lanes
// of a chunk holds consecutive row-order entries, so the row of (lane, slot
// j) is 4 * (sum over the chunk's slots before j of all their (run + 1))
// + 4 * (sum of slot j's (run + 1) over the chunk's lanes up to this one)
// - 4, from the chunk's start; a chunk that goes on from the previous pass
// starts at carry4.  The eight slot sums are four wavefront scans of 16-bit
// pairs (each field at most 64 * 64 = 4096), read back at the chunk's head
// and last lane through LDS.  Returns the segment-relative end of the chunk
// of lane last_lane (the pass's last group: the next pass's carry when its
// segment goes on), wavefront-uniform.
__device__ __forceinline__ int accumulate_pass_il(const PassIl& a, int carry4, int base4_cap, uint32_t tile_lds,
                                                  int* scr, int lane, int last_lane) {
  const uint32_t rw = a.live ? a.rw : 0u;
  const uint32_t E = rw & 0x0F0F0F0Fu, O = (rw >> 4) & 0x0F0F0F0Fu;   // bytes: runs of slots 0,2,4,6 / 1,3,5,7
  // pair q: slot 2q in bits 0..15, slot 2q + 1 in bits 16..31, each 4 * (run + 1)
  const uint32_t live4 = a.live ? 0x00040004u : 0u;
  uint32_t P[4];
  P[0] = (__builtin_amdgcn_perm(O, E, 0x0C040C00u) << 2) + live4;
  P[1] = (__builtin_amdgcn_perm(O, E, 0x0C050C01u) << 2) + live4;
  P[2] = (__builtin_amdgcn_perm(O, E, 0x0C060C02u) << 2) + live4;
  P[3] = (__builtin_amdgcn_perm(O, E, 0x0C070C03u) << 2) + live4;
  uint4 S;
  S.x = static_cast<uint32_t>(wave_inclusive_scan(static_cast<int>(P[0])));
  S.y = static_cast<uint32_t>(wave_inclusive_scan(static_cast<int>(P[1])));
  S.z = static_cast<uint32_t>(wave_inclusive_scan(static_cast<int>(P[2])));
  S.w = static_cast<uint32_t>(wave_inclusive_scan(static_cast<int>(P[3])));
  uint4* scr4 = reinterpret_cast<uint4*>(scr);
  scr4[lane] = S;
  wave_lds_sync();
  const uint4 Xh = a.hl > 0 ? scr4[a.hl - 1] : make_uint4(0u, 0u, 0u, 0u);   // before the chunk's head
  const uint4 Z = scr4[a.el];                                               // through its last lane
  // no field borrows: the scans are non-decreasing in every field
  const uint32_t I0 = S.x - Xh.x, I1 = S.y - Xh.y, I2 = S.z - Xh.z, I3 = S.w - Xh.w;
  const uint32_t T0 = Z.x - Xh.x, T1 = Z.y - Xh.y, T2 = Z.z - Xh.z, T3 = Z.w - Xh.w;
  // slot bases: the chunk's totals of the slots before each
  const uint32_t b1 = T0 & 0xFFFFu, b2 = b1 + (T0 >> 16), b3 = b2 + (T1 & 0xFFFFu), b4 = b3 + (T1 >> 16);
  const uint32_t b5 = b4 + (T2 & 0xFFFFu), b6 = b5 + (T2 >> 16), b7 = b6 + (T3 & 0xFFFFu), span = b7 + (T3 >> 16);
  // base + index sums per pair (fields below 8 * 4096 = 2^15: no carry)
  const uint32_t Q0 = I0 + (b1 << 16), Q1 = I1 + (b2 | (b3 << 16)), Q2 = I2 + (b4 | (b5 << 16));
  const uint32_t Q3 = I3 + (b6 | (b7 << 16));
  const int cb4 = a.first ? 0 : carry4;
  if (a.live) {
    const float xs = a.xs;
    // entry address: the chunk's start - 4 + its field, capped to the tile's
    // slack (a corrupt stream stays inside the tile)
    const uint32_t base = static_cast<uint32_t>(cb4 - 4) + tile_lds;
    const uint32_t cap = static_cast<uint32_t>(base4_cap) + tile_lds;
    tile_add_at(min(add_word<0>(base, Q0), cap), round_to_fixed(mul_lo_f16(a.v.x, xs)));
    tile_add_at(min(add_word<1>(base, Q0), cap), round_to_fixed(mul_hi_f16(a.v.x, xs)));
    tile_add_at(min(add_word<0>(base, Q1), cap), round_to_fixed(mul_lo_f16(a.v.y, xs)));
    tile_add_at(min(add_word<1>(base, Q1), cap), round_to_fixed(mul_hi_f16(a.v.y, xs)));
    tile_add_at(min(add_word<0>(base, Q2), cap), round_to_fixed(mul_lo_f16(a.v.z, xs)));
    tile_add_at(min(add_word<1>(base, Q2), cap), round_to_fixed(mul_hi_f16(a.v.z, xs)));
    tile_add_at(min(add_word<0>(base, Q3), cap), round_to_fixed(mul_lo_f16(a.v.w, xs)));
    tile_add_at(min(add_word<1>(base, Q3), cap), round_to_fixed(mul_hi_f16(a.v.w, xs)));
  }
  return __builtin_amdgcn_readlane(cb4 + static_cast<int>(span), last_lane);
}

struct KernelArgs {
  const uint32_t* gptr;
  const uint4* values;          // 8 fp16 per uint4
  const uint32_t* runs;
  const unsigned short* x;      // fp16 bits
  unsigned short* y;            // fp16 bits
  unsigned long long* ws;       // [2M] merge words (see the merge below)
  const unsigned short* colmax; // [K] fp16 bits: largest |stored weight| of each column
  float tau;
  uint32_t n_groups;
  int M, K, R, Kc, KC;
};

// Up to kMaxBatch independent products in one launch: grid (max blocks, n),
// product blockIdx.y owns workgroups blockIdx.x < blocks[blockIdx.y].  (The
// product is found from the block index alone, so its arguments arrive with
// one scalar load latency, as for a single product.)
constexpr int kMaxBatch = 8;
struct BatchArgs {
  int blocks[kMaxBatch];
  KernelArgs prod[kMaxBatch];
};

// The arguments a workgroup's prologue needs (the selection's pointers and
// sizes, the column maxima, R and M; the LDS layout follows from R and Kc).  A single-product launch passes
// them as leading kernel arguments, which gfx950 preloads into scalar
// registers at dispatch (the library is built with
// -amdgpu-kernarg-preload-count), so neither the selection's first memory
// round trip nor the LDS initialisation waits for the argument block.
struct Early {
  const uint32_t* gptr;
  const unsigned short* x;
  const unsigned short* colmax;
  int K, Kc, KC;
  float tau;
  int R, M;
};

// One workgroup's share of product p: row tile and column slice number blk.
template <int WAVES, int G, int DEPTH, int VAR>
__device__ __forceinline__ void spmspv_block(const Early& e, const KernelArgs& p, int blk) {
  static_assert(VAR == kVarRlc || G == 1, "the other variants take one group per lane");
  constexpr int NT = WAVES * kWave;
  extern __shared__ __align__(16) unsigned char smem[];
  int* tile = reinterpret_cast<int*>(smem);
  // the tile's LDS byte address (for the accumulation's own LDS instructions)
  const uint32_t tile_lds = static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) unsigned char*)smem));
  const LdsLayout lay = lds_layout(e.R, e.Kc, WAVES, scr_words_of(G, VAR));
  SegInfo* seg = reinterpret_cast<SegInfo*>(smem + lay.seg_off);
  int* scr_all = reinterpret_cast<int*>(smem + lay.scr_off);
  uint32_t* part = reinterpret_cast<uint32_t*>(smem + lay.misc_off);   // 3*WAVES: the selection's scan

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const int t = blk / e.KC, c = blk - t * e.KC;

  // The selection's loads go first: they need only the leading (preloaded)
  // arguments, so the workgroup's first memory round trip does not wait for
  // the rest of its argument block or for the LDS initialisation.
  const int k0 = c * e.Kc;
  const int kn = min(e.Kc, e.K - k0);
  const uint32_t* gp = e.gptr + static_cast<size_t>(t) * e.K + k0;
  const bool one_per_lane = kn <= NT;   // workgroup-uniform
  uint32_t g[kMaxCols + 1], xr[kMaxCols], cm[kMaxCols];
  int m = 1, kb = tid;
  if (one_per_lane) {
    g[0] = g[1] = xr[0] = cm[0] = 0u;
    if (tid < kn) {
      g[0] = gp[tid];
      g[1] = gp[tid + 1];
      xr[0] = e.x[k0 + tid];
      cm[0] = e.colmax[k0 + tid];
    }
  } else {
    // m <= kMaxCols consecutive columns per lane; all kMaxCols slots are
    // loaded, at clamped indices and without branches, so that no load waits
    // for another (columns at or past kn, or past the lane's m, are dropped
    // by the keep test)
    m = (kn + NT - 1) / NT;
    kb = tid * m;
#pragma unroll
    for (int j = 0; j <= kMaxCols; ++j) g[j] = gp[min(kb + j, kn)];
#pragma unroll
    for (int j = 0; j < kMaxCols; ++j) xr[j] = e.x[k0 + min(kb + j, kn - 1)];
#pragma unroll
    for (int j = 0; j < kMaxCols; ++j) cm[j] = e.colmax[k0 + min(kb + j, kn - 1)];
  }

  const int row0 = t * e.R;
  const int rows = min(e.R, e.M - row0);
  const int base4_cap = 4 * (e.R + 7);   // tile byte address cap of a group base

  for (int i = tid; i < lay.tile_slots; i += NT) tile[i] = 0;
  for (int i = tid; i < NT * scr_words_of(G, VAR); i += NT) scr_all[i] = 0;
  int scale = 0;   // the workgroup's fixed-point scale 2^scale

  // ---- selection of this slice's active, non-empty columns ----------------
  // The flat group sequence is then cut into equal ranges, one per
  // wavefront (a segment may be shared by several).
  // B = n * max over the n kept columns of colmax[k] * |x_k| bounds the sum
  // of |products| of every row of the slice; the tile's grid 2^-scale puts B
  // just below 2^30 (the products' half-unit roundings stay far inside
  // int32).  Non-negative floats order like their bit patterns, so the
  // maximum is an integer scan.
  uint32_t n_seg, n_grp;
  if (one_per_lane) {
    // one column per lane
    const uint32_t g0 = g[0], g1 = g[1];
    const float xv = half_bits_to_float(xr[0]);
    const bool keep = tid < kn && fabsf(xv) > e.tau && g1 > g0;
    const uint32_t cnt = keep ? g1 - g0 : 0u;
    uint32_t en, eg, tmax;
    block_scan_select<WAVES>(keep ? 1u : 0u, cnt, keep ? __float_as_uint(fabsf(xv) * half_bits_to_float(cm[0])) : 0u,
                             en, eg, n_seg, n_grp, tmax, part);
    const int s = grid_scale(static_cast<float>(n_seg) * __uint_as_float(tmax), 30);
    if (keep) seg[en] = SegInfo{g0, eg, cnt, ldexpf(xv, s)};
    scale = s;
  } else {
    // m <= kMaxCols consecutive columns per lane (loaded above), so one block
    // scan still orders all of them: segment order is column order
    uint32_t keep_bits = 0u, n_loc = 0u, g_loc = 0u, m_loc = 0u;
#pragma unroll
    for (int j = 0; j < kMaxCols; ++j) {
      const float xv = half_bits_to_float(xr[j]);
      const bool keep = j < m && kb + j < kn && fabsf(xv) > e.tau && g[j + 1] > g[j];
      keep_bits |= (keep ? 1u : 0u) << j;
      n_loc += keep ? 1u : 0u;
      g_loc += keep ? g[j + 1] - g[j] : 0u;
      m_loc = max(m_loc, keep ? __float_as_uint(fabsf(xv) * half_bits_to_float(cm[j])) : 0u);
    }
    uint32_t en, eg, tmax;
    block_scan_select<WAVES>(n_loc, g_loc, m_loc, en, eg, n_seg, n_grp, tmax, part);
    const int s = grid_scale(static_cast<float>(n_seg) * __uint_as_float(tmax), 30);
    uint32_t idx = en, off = eg;
#pragma unroll
    for (int j = 0; j < kMaxCols; ++j) {
      if ((keep_bits >> j) & 1u) {
        const uint32_t cnt = g[j + 1] - g[j];
        seg[idx] = SegInfo{g[j], off, cnt, ldexpf(half_bits_to_float(xr[j]), s)};
        ++idx;
        off += cnt;
      }
    }
    scale = s;
  }
  __syncthreads();

  // ---- per-wavefront walk over passes of 64*G groups -----------------------
  // A ring of DEPTH passes is kept in flight: after a pass is decoded and
  // accumulated, its slot is refilled with the loads of the pass DEPTH ahead.
  // The ring is indexed by compile-time constants (fully unrolled), so no
  // register copies force an early wait.  Passes past the end are idle (every
  // lane inactive, loads of group 0) and accumulate nothing.
  constexpr uint32_t P = kWave * G;
  // Wavefront wv walks the flat groups [pb0, pe), starting in segment
  // i_begin.  Segments past the range are never assigned to a live lane, so
  // the walk's segment bound is simply n_seg.
  const int wvu = __builtin_amdgcn_readfirstlane(wv);
  if constexpr (VAR == kVarInterleaved) {
    // ranges and passes cut at chunk boundaries (the same function of the
    // equal cuts for every wavefront, so the ranges still tile the sequence)
    const uint32_t pb0 = chunk_boundary(seg, static_cast<int>(n_seg), n_grp, cut_of<WAVES>(wvu, n_grp), lane);
    const uint32_t pe = chunk_boundary(seg, static_cast<int>(n_seg), n_grp, cut_of<WAVES>(wvu + 1, n_grp), lane);
    if (pb0 < pe) {
      SegInfo s0;
      const int i_begin = holding_segment(seg, static_cast<int>(n_seg), pb0, lane, s0);
      const int i_end = static_cast<int>(n_seg);
      const Streams st = make_streams(p.values, p.runs, p.n_groups, 4u);
      int* scr = scr_all + wv * kWave * scr_words_of(G, VAR);
      PassIl ring[DEPTH];
      uint32_t pf = pb0;    // flat start of the next pass to fetch
      int icur = i_begin;   // segment holding group pf
#pragma unroll
      for (int d = 0; d < DEPTH; ++d) {
        fetch_pass_il(ring[d], st, seg, scr, pf, icur, i_end, pe, lane);
        icur = ring[d].next_seg;
        pf = ring[d].pend;
      }
      // a range that starts inside a segment starts after whole chunks of
      // it: their span is the sum of their groups' spans, in any order (read
      // while the ring's loads are in flight)
      const uint32_t before = pb0 - s0.off;
      int carry = 0;
      if (before > 0u) {
        int acc = 0;
        for (uint32_t j = lane; j - lane < before; j += kWave) {
          const uint32_t rw =
              __builtin_amdgcn_raw_buffer_load_b32(st.runs, static_cast<int>((s0.gstart + min(j, before - 1u)) << 2), 0, 0);
          acc += j < before ? group_span4(rw) : 0;
        }
        carry = __builtin_amdgcn_readlane(wave_inclusive_scan(acc), kWave - 1);
      }
      uint32_t pb = pb0;    // flat start of the pass being accumulated
      // wavefront-uniform; every pass holds at least one chunk, so pe - pb0
      // rounds of DEPTH passes are more than enough (the bound only makes
      // termination evident)
      for (uint32_t round = 0; pb < pe && round < pe - pb0; ++round) {
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
          if (pb < pe) {
            const int last_lane = static_cast<int>(ring[d].pend - 1u - pb);
            const int tail = accumulate_pass_il(ring[d], carry, base4_cap, tile_lds, scr, lane, last_lane);
            carry = ring[d].cont ? tail : 0;
            pb = ring[d].pend;
          }
          fetch_pass_il(ring[d], st, seg, scr, pf, icur, i_end, pe, lane);
          icur = ring[d].next_seg;
          pf = ring[d].pend;
        }
      }
    }
  } else {
    const uint32_t pb0 = cut_of<WAVES>(wvu, n_grp);
    const uint32_t pe = cut_of<WAVES>(wvu + 1, n_grp);
    if (pb0 < pe) {
      SegInfo s0;
      const int i_begin = holding_segment(seg, static_cast<int>(n_seg), pb0, lane, s0);
      const int i_end = static_cast<int>(n_seg);
      const Streams st = make_streams(p.values, p.runs, p.n_groups, VAR == kVarRows16 ? 16u : 4u);
      int* scr = scr_all + wv * kWave * scr_words_of(G, VAR);
      const int n_pass = static_cast<int>((pe - pb0 + P - 1) / P);
      // A range that starts inside a segment starts at the row reached by the
      // segment's earlier groups: their runs (up to 4 * 64 groups here, the
      // rest below) are loaded ahead of the ring, so that their round trip
      // overlaps the ring's.
      const uint32_t before = VAR == kVarRows16 ? 0u : pb0 - s0.off;   // row offsets need no start row
      uint32_t rb[4] = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (before > static_cast<uint32_t>(q * kWave)) {   // wavefront-uniform
          // lanes past the earlier groups reread the last of them (their own
          // lines, not one line shared by every wavefront)
          const uint32_t j = min(static_cast<uint32_t>(q * kWave + lane), before - 1u);
          rb[q] = __builtin_amdgcn_raw_buffer_load_b32(st.runs, static_cast<int>((s0.gstart + j) << 2), 0, 0);
        }
      }
      Pass<G> ring[DEPTH];
      const uint32_t cap_rows2 = static_cast<uint32_t>(e.R + 7) * 0x00010001u;   // both halves: R + 7
      uint32_t pf = pb0;    // flat start of the next pass to fetch
      int icur = i_begin;   // segment holding group pf
#pragma unroll
      for (int d = 0; d < DEPTH; ++d) {
        fetch_pass<G, VAR == kVarRows16>(ring[d], st, seg, scr, pf, icur, i_end, pe, lane);
        icur = next_pass_segment<G>(ring[d], pf, i_end);
        pf += P;
      }
      uint32_t pb = pb0;    // flat start of the pass being accumulated
      int carry = 0;        // 4 * sum of (run + 1) over its first segment's earlier groups
      if (before > 0u) {
        int acc = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) acc += static_cast<uint32_t>(q * kWave + lane) < before ? group_span4(rb[q]) : 0;
        for (uint32_t j = 4 * kWave + lane; j - lane < before; j += kWave) {   // segments longer than 256 groups
          const uint32_t rw =
              __builtin_amdgcn_raw_buffer_load_b32(st.runs, static_cast<int>((s0.gstart + min(j, before - 1u)) << 2), 0, 0);
          acc += j < before ? group_span4(rw) : 0;
        }
        carry = __builtin_amdgcn_readlane(wave_inclusive_scan(acc), kWave - 1);
      }
      for (int done = 0; done < n_pass; done += DEPTH) {
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
          if (pb < pe) {   // wavefront-uniform
            if constexpr (VAR == kVarRows16) {
              accumulate_pass_rows16<G>(ring[d], cap_rows2, tile_lds);
            } else {
              const int tail = accumulate_pass<G, VAR == kVarSwizzle>(ring[d], carry, base4_cap, tile_lds, scr, lane);
              carry = ring[d].end63 > pb + P ? tail : 0;
            }
          }
          pb += P;
          fetch_pass<G, VAR == kVarRows16>(ring[d], st, seg, scr, pf, icur, i_end, pe, lane);
          icur = next_pass_segment<G>(ring[d], pf, i_end);
          pf += P;
        }
      }
    }
  }
  __syncthreads();

  // ---- merge --------------------------------------------------------------
  // the tile slot of row r
  const auto slot = [](int r) -> int {
    return VAR == kVarSwizzle ? static_cast<int>(swizzle4(4u * static_cast<uint32_t>(r)) >> 2) : r;
  };
  if (e.KC == 1) {
    for (int r = tid; r < rows; r += NT)
      p.y[row0 + r] = float_to_half_bits(ldexpf(static_cast<float>(tile[slot(r)]), -scale));
    return;
  }
  // Row r of the product owns two 64-bit words of the workspace: ws[r]
  // collects tickets, ws[M + r] the excesses.  Every slice adds one ticket
  // per row with a returning atomic: its partial p, clamped to +-4096, as a
  // multiple of 2^-33 (at most 2^45 in magnitude) plus a bias of 2^45 that
  // keeps it non-negative (bits 0..51), 1 in the arrival count (bits 58..63)
  // and, when p was clamped, 1 in the excess count (bits 52..57).  KC <= 63
  // slices keep each field from carrying into the next.  A slice whose p
  // exceeds the clamp first adds p minus the clamp, as a multiple of 2^-8, to
  // ws[M + r], and a release fence orders that add before the wavefront's
  // tickets.  The slice whose atomic returns count KC-1 holds the complete
  // sum of the clamped partials; when the excess count is non-zero it also
  // reads ws[M + r] (after an acquire fence).  It writes y[r] and clears the
  // words for the next call.
  // Per workgroup: a partial q (units of 2^-scale) is clamped iff |q| > lim,
  // i.e. |q * 2^-scale| > 4096; otherwise its ticket value is q * 2^(33 - scale)
  // (rounded, ties upward, when the tile's grid is finer than 2^-33).
  const int lim = scale >= 19 ? 0x7FFFFFFF : (scale >= -12 ? (1 << (scale + 12)) : 0);
  const int sh = 33 - scale;
  const auto fine_ticket = [&](int q) -> unsigned long long {
    const long long f = sh >= 0 ? static_cast<long long>(q) * (1ll << min(sh, 45))
                                : ((static_cast<long long>(q) + (1ll << (-sh - 1))) >> -sh);
    return kTicketCount + static_cast<unsigned long long>(f + kFineClamp);
  };
  // the excess of a clamped partial on the grid 2^-8 (scale < 19 here)
  const auto excess_of = [&](int q) -> long long {
    const int se = 8 - scale;
    const long long v = se >= 0 ? static_cast<long long>(q) * (1ll << min(se, 32))
                                : ((static_cast<long long>(q) + (1ll << (-se - 1))) >> -se);
    // beyond +-2^48 (so far past fp16's range that the row is +-inf either
    // way) the excess is clamped, so that 63 of them cannot overflow int64
    const long long ex = v - (q < 0 ? -(1ll << 20) : (1ll << 20)), cap = 1ll << 56;
    return ex < -cap ? -cap : (ex > cap ? cap : ex);
  };
  const auto finish_row = [&](int r, unsigned long long ticket, unsigned long long old) {
    const unsigned long long sum = old + ticket;
    if ((old >> 58) == static_cast<unsigned long long>(e.KC - 1)) {
      const long long fine = static_cast<long long>(sum & (kTicketExcess - 1)) -
                             static_cast<long long>(e.KC) * kFineClamp;
      float v = ldexpf(static_cast<float>(fine), -33);
      if ((sum >> 52) & 63ull) {   // rare: some slice's partial was clamped
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        const long long c = static_cast<long long>(
            __hip_atomic_load(p.ws + e.M + row0 + r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        v += ldexpf(static_cast<float>(c), -8);
        p.ws[e.M + row0 + r] = 0ull;
      }
      p.y[row0 + r] = float_to_half_bits(v);
      p.ws[row0 + r] = 0ull;
    }
  };
  // a lane's rows go J at a time (J = 1 when the tile has no more rows than
  // the workgroup has lanes, 2 up to twice that, else 4), their atomics
  // issued back to back under the execution mask (rows past a partial last
  // tile issue none: a shared dummy slot would serialise every such lane of
  // every slice on one address), then their returns are examined.  (The
  // fences sit in the rare branches: a fence acts for the whole wavefront.)
  const auto merge_rows = [&](auto in_flight) {
    constexpr int J = decltype(in_flight)::value;
    for (int r0 = tid; r0 - tid < rows; r0 += J * NT) {
      unsigned long long ticket[J], old[J];
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const int r = r0 + j * NT;
        const int q = r < rows ? tile[slot(r)] : 0;
        if ((q < 0 ? -q : q) <= lim) {
          ticket[j] = fine_ticket(q);
        } else {   // rare: the excess first, ordered before every ticket below
          atomicAdd(p.ws + e.M + row0 + r, static_cast<unsigned long long>(excess_of(q)));
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
          ticket[j] = kTicketCount + kTicketExcess +
                      static_cast<unsigned long long>((q < 0 ? -kFineClamp : kFineClamp) + kFineClamp);
        }
      }
#pragma unroll
      for (int j = 0; j < J; ++j) {
        old[j] = 0ull;
        if (r0 + j * NT < rows) old[j] = atomicAdd(p.ws + row0 + r0 + j * NT, ticket[j]);
      }
#pragma unroll
      for (int j = 0; j < J; ++j)
        if (r0 + j * NT < rows) finish_row(r0 + j * NT, ticket[j], old[j]);
    }
  };
  if (rows <= NT)
    merge_rows(std::integral_constant<int, 1>{});
  else if (rows <= 2 * NT)
    merge_rows(std::integral_constant<int, 2>{});
  else
    merge_rows(std::integral_constant<int, 4>{});
}

template <int WAVES, int G, int DEPTH, int VAR>
__global__ __launch_bounds__(WAVES * kWave) void spmspv_kernel(const uint32_t* gptr, const unsigned short* x,
                                                                const unsigned short* colmax, int K, int Kc, int KC,
                                                                float tau, int R, int M, KernelArgs p) {
  spmspv_block<WAVES, G, DEPTH, VAR>(Early{gptr, x, colmax, K, Kc, KC, tau, R, M}, p,
                                     static_cast<int>(blockIdx.x));
}

// (several products: the RLC layout and the plain tile only)
template <int WAVES, int G, int DEPTH>
__global__ __launch_bounds__(WAVES * kWave) void spmspv_batch_kernel(BatchArgs ba) {
  const int pi = static_cast<int>(blockIdx.y);
  if (static_cast<int>(blockIdx.x) >= ba.blocks[pi]) return;   // past this product's grid
  const KernelArgs& p = ba.prod[pi];
  spmspv_block<WAVES, G, DEPTH, kVarRlc>(Early{p.gptr, p.x, p.colmax, p.K, p.Kc, p.KC, p.tau, p.R, p.M},
                                         p, static_cast<int>(blockIdx.x));
}

// Zero-fills n bytes at p: the bytes before the first 8-byte boundary, then
// whole 64-bit words, then the rest.  A kernel rather than a memset, so that
// a caller may record it in a graph.
__global__ __launch_bounds__(256) void zero_fill_kernel(unsigned char* p, size_t n) {
  const size_t head = std::min(n, static_cast<size_t>((8u - (reinterpret_cast<uintptr_t>(p) & 7u)) & 7u));
  const size_t words = (n - head) / 8;
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  const size_t i0 = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  for (size_t i = i0; i < head; i += stride) p[i] = 0u;
  unsigned long long* w = reinterpret_cast<unsigned long long*>(p + head);
  for (size_t i = i0; i < words; i += stride) w[i] = 0ull;
  for (size_t i = head + 8 * words + i0; i < n; i += stride) p[i] = 0u;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Plan {
  int waves = 4, groups = 1, Kc = 0, KC = 0, T = 0, var = kVarRlc;
  int64_t blocks = 0;
  size_t lds = 0;
};

celty_status check_header(const celty_rlc_csc* W) {
  if (!W) return CELTY_EINVAL;
  if (W->version != CELTY_FORMAT_VERSION || W->run_bits != CELTY_RUN_BITS) return CELTY_EINVAL;
  if (W->layout != CELTY_LAYOUT_RLC && W->layout != CELTY_LAYOUT_ROWS16 && W->layout != CELTY_LAYOUT_INTERLEAVED)
    return CELTY_EINVAL;
  // 16-bit row offsets: four times R + 7 fits in 16 bits
  if (W->layout == CELTY_LAYOUT_ROWS16 && W->R > 16376) return CELTY_EINVAL;
  if (W->M < 1 || W->K < 1 || W->R < 1) return CELTY_EINVAL;
  if (W->T != static_cast<int32_t>((static_cast<int64_t>(W->M) + W->R - 1) / W->R)) return CELTY_EINVAL;
  if (W->n_groups < 0 || W->n_groups > static_cast<int64_t>(UINT32_MAX)) return CELTY_EINVAL;
  if (!W->gptr || misaligned(W->gptr, 4)) return CELTY_EINVAL;
  // buffer resources take byte sizes below 2^31
  if (W->n_groups * 16 > static_cast<int64_t>(INT32_MAX)) return CELTY_EINVAL;
  if (W->n_groups > 0 && (!W->values || !W->runs)) return CELTY_EINVAL;
  if (!(W->max_abs >= 0.f) || std::isinf(W->max_abs)) return CELTY_EINVAL;
  if (misaligned(W->values, 16) || misaligned(W->runs, W->layout == CELTY_LAYOUT_ROWS16 ? 16 : 4)) return CELTY_EINVAL;
  if (!W->colmax || misaligned(W->colmax, 4)) return CELTY_EINVAL;
  return CELTY_OK;
}

celty_status make_plan(const celty_rlc_csc* W, const celty_launch* cfg, Plan& pl) {
  if (celty_status st = check_header(W)) return st;
  pl.T = W->T;
  // automatic shape: 16 wavefronts per compute unit on 256 compute units,
  // as one workgroup of 16 (tiles of 1024 rows or more) or two of 8
  pl.waves = (cfg && cfg->waves_per_block) ? cfg->waves_per_block : (W->R >= 1024 ? 16 : 8);
  if (pl.waves != 2 && pl.waves != 4 && pl.waves != 8 && pl.waves != 16) return CELTY_EINVAL;
  int Kc = cfg ? cfg->cols_per_block : 0;
  if (Kc == 0) {
    // about 4096 / waves workgroups (16 wavefronts on each of 256 compute
    // units): T row tiles times KC slices (at most 63, the merge's count
    // byte) of a multiple of 64 columns
    const int64_t slots = 4096 / pl.waves;
    const int64_t kcs = std::min<int64_t>(kMaxSlices, std::max<int64_t>(1, (slots + W->T / 2) / W->T));
    int64_t kc = ((W->K + kcs - 1) / kcs + 63) / 64 * 64;
    const int64_t n_wg = W->T * ((W->K + kc - 1) / kc);
    // Counts past the slots start a second round, and 8-wavefront counts
    // between one and 0.9 x two per compute unit leave some units with two
    // and the rest with one.  Then, with no rounding of the width: slices
    // that would hold at least 80 KB of stored groups each at two workgroups
    // per unit take the most slices that fit the slots (two per unit);
    // lighter ones take one workgroup per unit, whose wider slices halve the
    // merge tickets (16 bytes per row and slice), which outweigh the second
    // workgroup's latency hiding on light slices.  Up to one workgroup per
    // unit the count is kept.
    const int64_t ks = std::min<int64_t>(kMaxSlices, std::max<int64_t>(1, slots / W->T));
    const bool uneven = pl.waves == 8 && n_wg > 256 && 10 * n_wg < 9 * slots;
    const double stored_per_wg = 20.0 * static_cast<double>(W->n_groups) / static_cast<double>(W->T * ks);
    if (n_wg > slots || (uneven && stored_per_wg >= 80.0 * 1024.0)) {
      kc = (W->K + ks - 1) / ks;
    } else if (uneven) {
      const int64_t k1 = std::min<int64_t>(kMaxSlices, std::max<int64_t>(1, 256 / W->T));
      kc = (W->K + k1 - 1) / k1;
    }
    kc = std::min<int64_t>(kc, std::min(4096, kMaxCols * kWave * pl.waves));
    Kc = static_cast<int>(kc);
  }
  if (Kc < 1 || Kc > 4096) return CELTY_EINVAL;
  if (Kc > W->K) Kc = W->K;
  if (Kc > kMaxCols * kWave * pl.waves) return CELTY_EINVAL;
  pl.Kc = Kc;
  pl.KC = (W->K + Kc - 1) / Kc;
  if (pl.KC > kMaxSlices) return CELTY_EINVAL;
  // one group per lane per pass unless asked otherwise: with several, the
  // lanes of one LDS add instruction land G groups apart, which costs more
  // bank conflicts than the bookkeeping it saves
  pl.groups = (cfg && cfg->groups_per_lane) ? cfg->groups_per_lane : 1;
  if (pl.groups != 1 && pl.groups != 2 && pl.groups != 4) return CELTY_EINVAL;
  // the variant: the layout's row encoding, or the swizzled tile (RLC only);
  // all but the plain RLC kernel take one group per lane
  const int swz = cfg ? cfg->lds_swizzle : 0;
  if (swz != 0 && swz != 1) return CELTY_EINVAL;
  if (W->layout == CELTY_LAYOUT_RLC)
    pl.var = swz ? kVarSwizzle : kVarRlc;
  else if (swz)
    return CELTY_EINVAL;
  else
    pl.var = W->layout == CELTY_LAYOUT_ROWS16 ? kVarRows16 : kVarInterleaved;
  if (pl.var != kVarRlc && pl.groups != 1) return CELTY_EINVAL;
  if (W->R > kMaxLds / 4) return CELTY_EINVAL;   // keeps the layout arithmetic in int
  pl.lds = static_cast<size_t>(lds_layout(W->R, pl.Kc, pl.waves, scr_words_of(pl.groups, pl.var)).bytes);
  if (pl.lds > static_cast<size_t>(kMaxLds)) return CELTY_EINVAL;
  pl.blocks = static_cast<int64_t>(W->T) * pl.KC;
  if (pl.blocks > 0x7FFFFFFF) return CELTY_EINVAL;
  return CELTY_OK;
}

// The launch: products, the largest per-product grid and LDS footprint.
struct Launch {
  int waves = 8, groups = 1, n = 0, var = kVarRlc;
  bool shallow = false;   // one group per lane with a ring of two passes instead of three
  int64_t max_blocks = 0;
  size_t lds = 0;
};

// Lets a kernel take more than 64 KB of dynamic LDS on the current device
// (once per kernel and device: `done` holds one bit per device id below 64;
// setting the attribute again is harmless, so two threads racing here are).
template <typename F>
bool allow_large_lds(F* fn, std::atomic<uint64_t>& done) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  const uint64_t bit = dev < 64 ? (1ull << dev) : 0ull;
  if (bit && (done.load(std::memory_order_relaxed) & bit)) return true;
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLds) !=
      hipSuccess)
    return false;
  done.fetch_or(bit, std::memory_order_relaxed);
  return true;
}

template <int WAVES, int G, int DEPTH, int VAR>
celty_status launch_shape(const Launch& ln, const BatchArgs& a, hipStream_t stream) {
  static std::atomic<uint64_t> single_attr{0}, batch_attr{0};
  if (ln.n == 1) {
    if (ln.lds > 64 * 1024 && !allow_large_lds(&spmspv_kernel<WAVES, G, DEPTH, VAR>, single_attr))
      return CELTY_EHIP;
    const KernelArgs& q = a.prod[0];
    hipLaunchKernelGGL((spmspv_kernel<WAVES, G, DEPTH, VAR>), dim3(static_cast<unsigned>(ln.max_blocks)),
                       dim3(WAVES * kWave), ln.lds, stream, q.gptr, q.x, q.colmax, q.K, q.Kc, q.KC, q.tau, q.R,
                       q.M, q);
  } else if constexpr (VAR == kVarRlc) {
    if (ln.lds > 64 * 1024 && !allow_large_lds(&spmspv_batch_kernel<WAVES, G, DEPTH>, batch_attr))
      return CELTY_EHIP;
    hipLaunchKernelGGL((spmspv_batch_kernel<WAVES, G, DEPTH>),
                       dim3(static_cast<unsigned>(ln.max_blocks), static_cast<unsigned>(ln.n)),
                       dim3(WAVES * kWave), ln.lds, stream, a);
  } else {
    return CELTY_EINVAL;   // rejected by celty_spmspv_batch before this point
  }
  return hipGetLastError() == hipSuccess ? CELTY_OK : CELTY_EHIP;
}

template <int WAVES, int VAR>
celty_status launch_depth(const Launch& ln, const BatchArgs& a, hipStream_t stream) {
  return ln.shallow ? launch_shape<WAVES, 1, 2, VAR>(ln, a, stream) : launch_shape<WAVES, 1, 3, VAR>(ln, a, stream);
}

template <int WAVES>
celty_status launch_groups(const Launch& ln, const BatchArgs& a, hipStream_t stream) {
  if (ln.var != kVarRlc) {
    if (ln.groups != 1 || ln.n != 1) return CELTY_EINVAL;
    switch (ln.var) {
      case kVarSwizzle: return launch_depth<WAVES, kVarSwizzle>(ln, a, stream);
      case kVarRows16: return launch_depth<WAVES, kVarRows16>(ln, a, stream);
      case kVarInterleaved: return launch_depth<WAVES, kVarInterleaved>(ln, a, stream);
      default: return CELTY_EINVAL;
    }
  }
  switch (ln.groups) {
    case 1: return launch_depth<WAVES, kVarRlc>(ln, a, stream);
    case 2: return launch_shape<WAVES, 2, 2, kVarRlc>(ln, a, stream);
    case 4: return launch_shape<WAVES, 4, 2, kVarRlc>(ln, a, stream);
    default: return CELTY_EINVAL;
  }
}

celty_status launch(const Launch& ln, const BatchArgs& a, hipStream_t stream) {
  switch (ln.waves) {
    case 2: return launch_groups<2>(ln, a, stream);
    case 4: return launch_groups<4>(ln, a, stream);
    case 8: return launch_groups<8>(ln, a, stream);
    case 16: return launch_groups<16>(ln, a, stream);
    default: return CELTY_EINVAL;
  }
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
  return pa < pb + nb && pb < pa + na;
}

// Validates one product's pointers and fills its kernel arguments.
celty_status product_args(const celty_rlc_csc* W, const Plan& pl, const void* x, float tau, void* y, void* ws,
                          KernelArgs& a) {
  if (!x || !y || misaligned(x, 2) || misaligned(y, 2) || std::isnan(tau)) return CELTY_EINVAL;
  if (overlaps(x, 2u * static_cast<size_t>(W->K), y, 2u * static_cast<size_t>(W->M))) return CELTY_EINVAL;
  a.gptr = W->gptr;
  a.values = reinterpret_cast<const uint4*>(W->values);
  a.runs = W->runs;
  a.x = static_cast<const unsigned short*>(x);
  a.y = static_cast<unsigned short*>(y);
  a.ws = static_cast<unsigned long long*>(ws);
  a.colmax = W->colmax;
  a.tau = tau;
  a.n_groups = static_cast<uint32_t>(W->n_groups);
  a.M = W->M;
  a.K = W->K;
  a.R = W->R;
  a.Kc = pl.Kc;
  a.KC = pl.KC;
  return CELTY_OK;
}

// The merge words of celty_spmspv_noalloc: a file-scope device array (one
// copy on every GPU the library runs on, held until the process ends) in
// place of a caller workspace.  Zero at load, zero-filled again by the first
// call on each device, and left zero by every completed call.
constexpr size_t kScratchBytes = size_t(2) << 20;   // two 64-bit words per row: M <= 131072
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on the current device.  In host code the
// array's name is only a stand-in for the symbol; its device address comes
// from hipGetSymbolAddress, taken once per device (with that device current)
// and kept.  The first call on a device also zero-fills the array on the
// caller's stream (a kernel, so it may be recorded in a graph).
std::mutex scratch_mutex;
void* scratch_address[64] = {};

celty_status scratch_on_current_device(hipStream_t stream, void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return CELTY_EHIP;
  if (dev < 0 || dev >= 64) return CELTY_EHIP;
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (!scratch_address[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return CELTY_EHIP;
    hipLaunchKernelGGL(zero_fill_kernel, dim3(static_cast<unsigned>(kScratchBytes / 8 / 256)), dim3(256), 0, stream,
                       static_cast<unsigned char*>(ptr), kScratchBytes);
    if (hipGetLastError() != hipSuccess) return CELTY_EHIP;
    scratch_address[dev] = ptr;
  }
  *out = scratch_address[dev];
  return CELTY_OK;
}

}  // namespace

extern "C" celty_status celty_spmspv_noalloc(const celty_rlc_csc* W, const void* x, float tau, void* y,
                                             const celty_launch* launch_cfg, void* stream) {
  if (celty_status st = check_header(W)) return st;
  const size_t need = celty_spmspv_workspace_bytes(W->M, W->K, W->R);
  if (need > kScratchBytes) return CELTY_EINVAL;   // more rows than the static array holds
  void* ws = nullptr;
  if (celty_status st = scratch_on_current_device(static_cast<hipStream_t>(stream), &ws)) return st;
  return celty_spmspv_batch(1, &W, &x, &tau, &y, ws, need, launch_cfg, stream);
}

extern "C" int32_t celty_default_tile_rows(int32_t M, int32_t K) {
  if (M < 1) return 0;
  // wide matrices (K >= 4M) take tiles twice as tall: their merge traffic,
  // which grows with M times the slices per tile, stays small next to the
  // data, and the longer segments stream better
  const int64_t span = static_cast<int64_t>(K) >= 4 * static_cast<int64_t>(M) ? M / 4 : M / 8;
  int32_t r = 256;
  while (r < 2048 && 2 * r <= span) r *= 2;
  return r;
}

extern "C" size_t celty_spmspv_workspace_bytes(int32_t M, int32_t K, int32_t R) {
  (void)K;
  (void)R;
  if (M < 1) return 0;
  return align_up(static_cast<size_t>(M) * 16, 256);
}

extern "C" celty_status celty_spmspv_workspace_init(void* workspace, size_t workspace_bytes, void* stream) {
  if (!workspace || workspace_bytes == 0) return CELTY_EINVAL;
  const size_t words = workspace_bytes / 8 + 1;
  const unsigned blocks = static_cast<unsigned>(std::min<size_t>((words + 255) / 256, 1024));
  hipLaunchKernelGGL(zero_fill_kernel, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<unsigned char*>(workspace), workspace_bytes);
  return hipGetLastError() == hipSuccess ? CELTY_OK : CELTY_EHIP;
}

extern "C" celty_status celty_spmspv_plan(const celty_rlc_csc* W, const celty_launch* launch_cfg,
                                          celty_launch* resolved, int64_t* n_blocks, int64_t* lds_bytes) {
  if (!resolved) return CELTY_EINVAL;
  Plan pl;
  if (celty_status st = make_plan(W, launch_cfg, pl)) return st;
  resolved->cols_per_block = pl.Kc;
  resolved->waves_per_block = pl.waves;
  resolved->groups_per_lane = pl.groups;
  resolved->lds_swizzle = pl.var == kVarSwizzle ? 1 : 0;
  if (n_blocks) *n_blocks = pl.blocks;
  if (lds_bytes) *lds_bytes = static_cast<int64_t>(pl.lds);
  return CELTY_OK;
}

extern "C" celty_status celty_spmspv_ex(const celty_rlc_csc* W, const void* x, float tau, void* y,
                                        void* workspace, size_t workspace_bytes, const celty_launch* launch_cfg,
                                        void* stream) {
  return celty_spmspv_batch(1, &W, &x, &tau, &y, workspace, workspace_bytes, launch_cfg, stream);
}

extern "C" size_t celty_spmspv_batch_workspace_bytes(int32_t n, const celty_rlc_csc* const* W) {
  if (n < 1 || n > kMaxBatch || !W) return 0;
  size_t total = 0;
  for (int i = 0; i < n; ++i) {
    if (!W[i]) return 0;
    total += celty_spmspv_workspace_bytes(W[i]->M, W[i]->K, W[i]->R);
  }
  return total;
}

extern "C" celty_status celty_spmspv_batch(int32_t n, const celty_rlc_csc* const* W, const void* const* x,
                                           const float* tau, void* const* y, void* workspace,
                                           size_t workspace_bytes, const celty_launch* launch_cfg, void* stream) {
  if (n < 1 || n > kMaxBatch || !W || !x || !tau || !y) return CELTY_EINVAL;
  for (int i = 0; i < n; ++i)
    if (celty_status st = check_header(W[i])) return st;
  // one wavefront count and group count for the whole launch
  Launch ln;
  if (launch_cfg && launch_cfg->waves_per_block) {
    ln.waves = launch_cfg->waves_per_block;
  } else {
    ln.waves = 8;
    for (int i = 0; i < n; ++i)
      if (W[i]->R >= 1024) ln.waves = 16;
  }
  ln.groups = (launch_cfg && launch_cfg->groups_per_lane) ? launch_cfg->groups_per_lane : 1;
  const celty_launch cfg{launch_cfg ? launch_cfg->cols_per_block : 0, ln.waves, ln.groups,
                         launch_cfg ? launch_cfg->lds_swizzle : 0};
  const size_t need = celty_spmspv_batch_workspace_bytes(n, W);
  if (!workspace || misaligned(workspace, 256) || workspace_bytes < need) return CELTY_EINVAL;

  BatchArgs ba{};
  ln.n = n;
  int64_t total_blocks = 0;
  double stored_groups = 0.0;
  size_t ws_off = 0;
  for (int i = 0; i < n; ++i) {
    Plan pl;
    if (celty_status st = make_plan(W[i], &cfg, pl)) return st;
    // the swizzled tile and the other layouts run one product per launch
    if (n > 1 && pl.var != kVarRlc) return CELTY_EINVAL;
    ln.var = pl.var;
    void* ws_i = static_cast<unsigned char*>(workspace) + ws_off;
    if (celty_status st = product_args(W[i], pl, x[i], tau[i], y[i], ws_i, ba.prod[i])) return st;
    ws_off += celty_spmspv_workspace_bytes(W[i]->M, W[i]->K, W[i]->R);
    ba.blocks[i] = static_cast<int>(pl.blocks);   // make_plan keeps it below 2^31
    ln.max_blocks = std::max(ln.max_blocks, pl.blocks);
    ln.lds = std::max(ln.lds, pl.lds);
    total_blocks += pl.blocks;
    stored_groups += static_cast<double>(W[i]->n_groups);
  }
  // every y is written while the other products read their x; none may
  // overlap another product's x or y, or the workspace
  for (int i = 0; i < n; ++i) {
    const size_t yb = 2u * static_cast<size_t>(W[i]->M);
    if (overlaps(y[i], yb, workspace, need)) return CELTY_EINVAL;
    if (overlaps(x[i], 2u * static_cast<size_t>(W[i]->K), workspace, need)) return CELTY_EINVAL;
    for (int j = 0; j < n; ++j) {
      if (j == i) continue;
      if (overlaps(y[i], yb, x[j], 2u * static_cast<size_t>(W[j]->K))) return CELTY_EINVAL;
      if (overlaps(y[i], yb, y[j], 2u * static_cast<size_t>(W[j]->M))) return CELTY_EINVAL;
    }
  }
  // Ring depth: with two 8-wavefront workgroups on a compute unit, two passes
  // in flight per wavefront suffice, and walks of a few to a dozen passes
  // run faster with two than with three; one workgroup per unit, and
  // 16-wavefront workgroups, keep three.  The pass count is estimated with
  // half of the stored groups active (the activation is not known here).
  const double passes =
      total_blocks > 0 ? 0.5 * stored_groups / (static_cast<double>(total_blocks) * ln.waves * kWave) : 0.0;
  ln.shallow = ln.groups == 1 && ln.waves == 8 && total_blocks > 256 && passes >= 4.0 && passes <= 16.0;
  return launch(ln, ba, static_cast<hipStream_t>(stream));
}

extern "C" celty_status celty_spmspv(const celty_rlc_csc* W, const void* x, float tau, void* y, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  return celty_spmspv_ex(W, x, tau, y, workspace, workspace_bytes, nullptr, stream);
}

extern "C" const char* celty_status_string(celty_status status) {
  switch (status) {
    case CELTY_OK: return "CELTY_OK: success";
    case CELTY_EINVAL: return "CELTY_EINVAL: invalid argument";
    case CELTY_ENOMEM: return "CELTY_ENOMEM: host scratch or worker threads unavailable";
    case CELTY_EOVERFLOW: return "CELTY_EOVERFLOW: group count exceeds uint32";
    case CELTY_EFORMAT: return "CELTY_EFORMAT: malformed RLC-CSC stream";
    case CELTY_EHIP: return "CELTY_EHIP: HIP runtime error";
  }
  return "unknown celty_status";
}
