// One-shot magnitude pruning of one fp16/bf16 matrix (paper section 2 removes
// the weights of smallest magnitude before sparse training): the keep-mask
// zeroes exactly `prune` entries, those of smallest |w|, ties in ascending
// row-major index.
//
// For non-NaN fp16/bf16 payloads the order of |w| is the order of the 15-bit
// key bits & 0x7fff, and equal keys are equal magnitudes (+0 and -0 share key
// 0).  Three passes over the keys:
//   1. a 32768-bin histogram (per-workgroup LDS histograms added into HBM);
//   2. one workgroup scans it for the threshold key T (the smallest key whose
//      cumulative count reaches `prune`) and `need`, the number of entries
//      equal to T that are zeroed (prune minus the count below T);
//   3. per chunk of the matrix, the number of entries equal to T; then each
//      workgroup ranks its T entries in index order (the counts of earlier
//      chunks plus a workgroup scan) and writes the mask: key < T -> 0,
//      key > T -> 1, key == T -> 0 iff rank < need.
#include "spl_common.h"

namespace spl {
namespace {

constexpr int kBins = 1 << 15;
constexpr int kPrThreads = 1024;
constexpr int kPrRound = 8 * kPrThreads;      // keys per workgroup round: one 16-byte load per thread
constexpr int kPrMaxChunks = 2048;

__device__ __forceinline__ uint32_t key_of(const u32x4& v, int e) { return (v[e >> 1] >> (16 * (e & 1))) & 0x7fffu; }

// Sum of x over the workgroup, and (exclusive) the sum over lower threads.
__device__ __forceinline__ uint32_t block_scan(uint32_t x, uint32_t* part, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t inc = wave_inclusive_scan(x);
  __syncthreads();                                   // part is free (earlier readers are done)
  if (lane == 63) part[wave] = inc;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kPrThreads / 64; ++w) {
    const uint32_t p = part[w];
    before += w < wave ? p : 0u;
    all += p;
  }
  *total = all;
  return before + inc - x;
}

__global__ void __launch_bounds__(kPrThreads) k_mag_hist(const uint16_t* __restrict__ W, int64_t n, int64_t chunk,
                                                         uint32_t* __restrict__ hist) {
  extern __shared__ uint32_t h[];                    // kBins counters
  for (int b = threadIdx.x; b < kBins; b += kPrThreads) h[b] = 0u;
  __syncthreads();
  const int64_t beg = (int64_t)blockIdx.x * chunk;
  const int64_t end = beg + chunk < n ? beg + chunk : n;
  for (int64_t i = beg + 8 * (int64_t)threadIdx.x; i < end; i += kPrRound) {   // chunk, n: multiples of 8
    const u32x4 v = *reinterpret_cast<const u32x4*>(W + i);
#pragma unroll
    for (int e = 0; e < 8; ++e) atomicAdd(&h[key_of(v, e)], 1u);
  }
  __syncthreads();
  for (int b = threadIdx.x; b < kBins; b += kPrThreads)
    if (h[b]) atomicAdd(&hist[b], h[b]);
}

// One workgroup: thread t owns bins [32t, 32t + 32).  sel[0] = T (0xffffffff:
// nothing is pruned), sel[1] = need.
__global__ void __launch_bounds__(kPrThreads) k_mag_select(const uint32_t* __restrict__ hist, uint32_t prune,
                                                           uint32_t* __restrict__ sel) {
  __shared__ uint32_t part[kPrThreads / 64];
  constexpr int BPT = kBins / kPrThreads;
  const int t = threadIdx.x;
  uint32_t s = 0;
#pragma unroll 8
  for (int j = 0; j < BPT; ++j) s += hist[BPT * t + j];
  uint32_t total;
  const uint32_t before = block_scan(s, part, &total);
  if (prune == 0u) {
    if (t == 0) sel[0] = 0xffffffffu, sel[1] = 0u;
  } else if (before < prune && prune <= before + s) {     // exactly one thread: prune <= n = total
    uint32_t run = before;
    for (int j = 0; j < BPT; ++j) {
      const uint32_t c = hist[BPT * t + j];
      if (run + c >= prune) {
        sel[0] = (uint32_t)(BPT * t + j);
        sel[1] = prune - run;
        break;
      }
      run += c;
    }
  }
}

__global__ void __launch_bounds__(kPrThreads) k_mag_ties(const uint16_t* __restrict__ W, int64_t n, int64_t chunk,
                                                         const uint32_t* __restrict__ sel, uint32_t* __restrict__ ties) {
  __shared__ uint32_t part[kPrThreads / 64];
  const uint32_t T = sel[0];
  const int64_t beg = (int64_t)blockIdx.x * chunk;
  const int64_t end = beg + chunk < n ? beg + chunk : n;
  uint32_t c = 0;
  for (int64_t i = beg + 8 * (int64_t)threadIdx.x; i < end; i += kPrRound) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(W + i);
#pragma unroll
    for (int e = 0; e < 8; ++e) c += key_of(v, e) == T ? 1u : 0u;
  }
  uint32_t total;
  (void)block_scan(c, part, &total);
  if (threadIdx.x == 0) ties[blockIdx.x] = total;
}

__global__ void __launch_bounds__(kPrThreads) k_mag_mask(const uint16_t* __restrict__ W, int64_t n, int64_t chunk,
                                                         const uint32_t* __restrict__ sel,
                                                         const uint32_t* __restrict__ ties,
                                                         uint8_t* __restrict__ mask) {
  __shared__ uint32_t part[kPrThreads / 64];
  const uint32_t T = sel[0], need = sel[1];
  uint32_t mine = 0;                                 // entries equal to T in earlier chunks
  for (int c = threadIdx.x; c < (int)blockIdx.x; c += kPrThreads) mine += ties[c];
  uint32_t run;
  (void)block_scan(mine, part, &run);
  const int64_t beg = (int64_t)blockIdx.x * chunk;
  const int64_t end = beg + chunk < n ? beg + chunk : n;
  for (int64_t r = beg; r < end; r += kPrRound) {    // uniform rounds: every thread reaches the scans
    const int64_t i = r + 8 * (int64_t)threadIdx.x;
    const bool live = i < end;
    u32x4 v = u32x4{0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu};   // key 0x7fff: never T below
    if (live) v = *reinterpret_cast<const u32x4*>(W + i);
    uint32_t cnt = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) cnt += (live && key_of(v, e) == T) ? 1u : 0u;
    uint32_t total;
    uint32_t rank = run + block_scan(cnt, part, &total);
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t k = key_of(v, e);
      uint32_t keep;
      if (k == T) {
        keep = rank >= need ? 1u : 0u;
        ++rank;
      } else {
        keep = (T == 0xffffffffu || k > T) ? 1u : 0u;
      }
      if (e < 4) lo |= keep << (8 * e);
      else hi |= keep << (8 * (e - 4));
    }
    if (live) *reinterpret_cast<u32x2*>(mask + i) = u32x2{lo, hi};
    run += total;
  }
}

}  // namespace

int64_t magnitude_mask_workspace_words() { return (int64_t)kBins + 2 + kPrMaxChunks; }

hipError_t launch_magnitude_mask(const uint16_t* W, int64_t n, uint32_t prune, uint8_t* mask, uint32_t* ws,
                                 hipStream_t s) {
  uint32_t* hist = ws;
  uint32_t* sel = ws + kBins;
  uint32_t* ties = ws + kBins + 2;
  int64_t chunks = (n + 65535) / 65536;
  if (chunks > kPrMaxChunks) chunks = kPrMaxChunks;
  if (chunks < 1) chunks = 1;
  const int64_t chunk = ((n + chunks - 1) / chunks + 7) / 8 * 8;
  chunks = (n + chunk - 1) / chunk;
  hipError_t e = launch_zero_fill(hist, 2 * kBins, s);
  if (e != hipSuccess) return e;
  static PerDeviceFlag lds_set;
  const hipError_t attr = allow_lds_once(lds_set, k_mag_hist, kBins * sizeof(uint32_t));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(k_mag_hist, dim3((unsigned)chunks), dim3(kPrThreads), kBins * sizeof(uint32_t), s, W, n, chunk,
                     hist);
  hipLaunchKernelGGL(k_mag_select, dim3(1), dim3(kPrThreads), 0, s, hist, prune, sel);
  hipLaunchKernelGGL(k_mag_ties, dim3((unsigned)chunks), dim3(kPrThreads), 0, s, W, n, chunk, sel, ties);
  hipLaunchKernelGGL(k_mag_mask, dim3((unsigned)chunks), dim3(kPrThreads), 0, s, W, n, chunk, sel, ties, mask);
  return hipGetLastError();
}

}  // namespace spl
