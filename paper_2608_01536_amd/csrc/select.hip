// Active-column selection kernels for gfx950 and their C ABI entry point,
// celty_select (Sections 1, 2.1 and 3.1: magnitude threshold, then stream
// compaction with wavefront ballots and prefix sums).  The SpMSpV kernels do
// the same selection inside their own prologue; this entry point gives the
// ascending list of active columns on its own.

#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>

#include "celty.h"
#include "common.h"

namespace {

// Global selection, one workgroup of 1024 lanes.
//
// select_kernel (x 4-byte aligned): x is taken in chunks of kSelSteps * 2048
// columns; in a chunk, lane tid of step j holds the two columns
// 2 * (j * 1024 + tid) + {0, 1}, read with one 32-bit buffer load (columns past
// K read as zero: the buffer's size is x's, rounded up to whole words).  All of
// a chunk's loads are issued before any is used and the lane keeps its
// activity bits in one register.  The wavefront totals of every (step,
// wavefront) pair go to LDS; after the chunk's one barrier every wavefront
// scans all pairs itself (in column order), so the offsets of its own pairs
// need no second barrier; within a pair, the ballots of the lanes' first and
// second columns give each active column its position.
//
// select_kernel_any (x only 2-byte aligned, or K <= 1024): steps of 1024
// columns, one column per lane, ranks from a ballot, two barriers per step.
constexpr int kSelSteps = 16;

__global__ __launch_bounds__(1024) void select_kernel(const unsigned short* __restrict__ x, int K, float tau,
                                                      int32_t* __restrict__ idx, int32_t* __restrict__ count) {
  constexpr int NW = 1024 / kWave;              // 16 wavefronts
  constexpr int PPL = kSelSteps * NW / kWave;   // pairs per lane in the scan (4)
  static_assert(PPL * kWave == kSelSteps * NW && NW % PPL == 0 && 2 * kSelSteps <= 32, "pair layout");
  __shared__ uint32_t cnt[kSelSteps * NW];      // pair (j, w) at j * NW + w: column order
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const __amdgpu_buffer_rsrc_t xs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<unsigned short*>(x), static_cast<short>(0), static_cast<int>((static_cast<uint32_t>(K) * 2u + 3u) & ~3u),
      0x00020000);
  uint32_t base = 0;
  for (int it = 0; it < K; it += kSelSteps * 2048) {
    const int steps = min(kSelSteps, (K - it + 2047) / 2048);   // workgroup-uniform
    uint32_t w[kSelSteps];
#pragma unroll
    for (int j = 0; j < kSelSteps; ++j)
      w[j] = __builtin_amdgcn_raw_buffer_load_b32(xs, (it + 2 * (j * 1024 + tid)) * 2, 0, 0);
    uint32_t bits = 0;   // bits 2j, 2j+1: the lane's two columns of step j
#pragma unroll
    for (int j = 0; j < kSelSteps; ++j) {
      if (j < steps) {
        const int k = it + 2 * (j * 1024 + tid);
        const bool a0 = k < K && fabsf(half_bits_to_float(w[j] & 0xFFFFu)) > tau;
        const bool a1 = k + 1 < K && fabsf(half_bits_to_float(w[j] >> 16)) > tau;
        bits |= ((a0 ? 1u : 0u) | (a1 ? 2u : 0u)) << (2 * j);
        const uint32_t tot = static_cast<uint32_t>(__popcll(__ballot(a0)) + __popcll(__ballot(a1)));
        if (lane == 0) cnt[j * NW + wv] = tot;
      }
    }
    __syncthreads();
    // every wavefront: lane l sums pairs PPL*l .. PPL*l + PPL-1 (those of
    // steps past the chunk's count as zero) and one wavefront scan orders them
    uint32_t c[PPL], lsum = 0;
#pragma unroll
    for (int i = 0; i < PPL; ++i) {
      const int pidx = PPL * lane + i;
      c[i] = pidx < steps * NW ? cnt[pidx] : 0u;
      lsum += c[i];
    }
    const uint32_t incl = static_cast<uint32_t>(wave_inclusive_scan(static_cast<int>(lsum)));
    const uint32_t total = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(incl), kWave - 1));
    // this wavefront's pair (j, wv) is slot wv % PPL of lane (j * NW + wv) / PPL
    const int slot = wv % PPL;
    uint32_t pre = incl - lsum;
#pragma unroll
    for (int i = 0; i < PPL; ++i) pre += i < slot ? c[i] : 0u;
    for (int j = 0; j < steps; ++j) {
      const int src = __builtin_amdgcn_readfirstlane((j * NW + wv) / PPL);
      const uint32_t o = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(pre), src));
      const bool a0 = (bits >> (2 * j)) & 1u, a1 = (bits >> (2 * j + 1)) & 1u;
      // columns of the lanes below come first: both of theirs, then this lane's
      const uint32_t e = base + o + lanes_below(__ballot(a0)) + lanes_below(__ballot(a1));
      const int k = it + 2 * (j * 1024 + tid);
      if (a0) idx[e] = k;
      if (a1) idx[e + (a0 ? 1u : 0u)] = k + 1;
    }
    base += total;
    if (it + kSelSteps * 2048 < K) __syncthreads();   // cnt[] is rewritten by the next chunk
  }
  if (tid == 0) *count = static_cast<int32_t>(base);
}

__global__ __launch_bounds__(1024) void select_kernel_any(const unsigned short* __restrict__ x, int K, float tau,
                                                          int32_t* __restrict__ idx, int32_t* __restrict__ count) {
  constexpr int NW = 1024 / kWave;
  __shared__ uint32_t wsum[NW];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  uint32_t base = 0;
  for (int it = 0; it < K; it += 1024) {
    const int k = it + tid;
    const bool act = k < K && fabsf(half_bits_to_float(x[k])) > tau;
    const uint64_t m = __ballot(act);
    const uint32_t rank = lanes_below(m);
    if (lane == 0) wsum[wv] = static_cast<uint32_t>(__popcll(m));
    __syncthreads();
    uint32_t off = base, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint32_t cw = wsum[w];
      if (w < wv) off += cw;
      tot += cw;
    }
    if (act) idx[off + rank] = k;
    base += tot;
    __syncthreads();
  }
  if (tid == 0) *count = static_cast<int32_t>(base);
}

}  // namespace

extern "C" celty_status celty_select(const void* x, int32_t K, float tau, int32_t* idx, int32_t* count,
                                     void* stream) {
  if (!x || !idx || !count || K < 1 || std::isnan(tau)) return CELTY_EINVAL;
  if (K > (INT32_MAX - 3) / 2) return CELTY_EINVAL;   // x's byte size is a 32-bit buffer size
  if (misaligned(x, 2) || misaligned(idx, 4) || misaligned(count, 4)) return CELTY_EINVAL;
  // word loads need x 4-byte aligned (the buffer ends at x's last word); up to
  // 1024 columns one step of the plain kernel is quicker
  if (K > 1024 && !misaligned(x, 4))
    hipLaunchKernelGGL(select_kernel, dim3(1), dim3(1024), 0, static_cast<hipStream_t>(stream),
                       static_cast<const unsigned short*>(x), K, tau, idx, count);
  else
    hipLaunchKernelGGL(select_kernel_any, dim3(1), dim3(1024), 0, static_cast<hipStream_t>(stream),
                       static_cast<const unsigned short*>(x), K, tau, idx, count);
  return hipGetLastError() == hipSuccess ? CELTY_OK : CELTY_EHIP;
}

