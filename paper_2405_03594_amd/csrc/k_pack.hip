// Bitmask-expansion encoder and decoder on gfx950 (paper section 2.4.1).
//
// pack_count : one wave per row counts kept entries, then one workgroup turns
//              the counts into exclusive row offsets (int64 running sums; an
//              overflow past 2^31 is flagged as row_offsets[N] = -1).
// pack_scatter: one wave per row walks the row in 64-column steps; a ballot of
//              the keep predicate is the row's next two bitmask words, and each
//              kept lane's rank among them (v_mbcnt) is its slot in `values`.
// unpack     : the inverse walk; a lane whose bit is set takes the value at its
//              rank, every other lane writes +0.
// retile16   : row layout -> tile layout (16 x 32 submatrices, paper section
//              2.4.2): per-tile counts and a scan give the tile offsets, then one
//              wave per row moves each word's values to their tile position.
// pack into the tile layout straight from W and the mask: per-tile counts and
//              the same scan, then one wave per tile, lane (row, column group)
//              in the order the tile stores its values, writes its kept values
//              at the exclusive wave scan of the lanes' counts and its byte(s) of
//              the row's bitmask word.
// validate   : the consistency of a compressed matrix (offsets against the
//              popcounts of the bitmask, first and last offsets, zero pad bits),
//              reported as error bits in a device word.
#include "spl_common.h"

namespace spl {
namespace {

template <int EB>
__device__ __forceinline__ bool payload_nonzero(const void* W, int64_t idx) {
  if constexpr (EB == 1) {
    return static_cast<const int8_t*>(W)[idx] != 0;
  } else {
    return (static_cast<const uint16_t*>(W)[idx] & 0x7fffu) != 0;   // -0.0 counts as zero
  }
}

template <int EB>
__device__ __forceinline__ bool is_kept(const void* W, const uint8_t* mask, int64_t idx) {
  return mask ? (mask[idx] != 0) : payload_nonzero<EB>(W, idx);
}

template <int EB>
__global__ void __launch_bounds__(256) k_row_count(const void* W, const uint8_t* mask, int64_t N, int64_t K,
                                                   int32_t* counts) {
  const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const uint32_t lane = threadIdx.x & 63u;
  const int64_t base = n * K;
  uint32_t c = 0;
  for (int64_t k = lane; k < K; k += kWave) c += is_kept<EB>(W, mask, base + k) ? 1u : 0u;
  for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
  if (lane == 0) counts[n] = (int32_t)c;
}

// In place: row_offsets[0..N) hold per-row counts on entry, exclusive prefix
// sums on exit; row_offsets[N] = nnz, or -1 if nnz >= 2^31 (then the other
// entries are left unspecified).  One workgroup walks the array in passes of
// 4096 entries: thread t takes four consecutive counts (one 16-byte load when
// the buffer is 16-byte aligned, so a pass's loads are coalesced), the waves
// scan their threads' sums with shuffles, the 16 wave totals go through LDS,
// and the pass's total is carried into the next pass.  A pass rewrites only
// the entries it has read.
__global__ void __launch_bounds__(1024) k_scan_offsets(int32_t* row_offsets, int64_t N) {
  __shared__ int64_t wsum[16];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const bool vec = ((uintptr_t)row_offsets & 15u) == 0;
  int64_t carry = 0;                                     // sum of every earlier pass
  for (int64_t base = 0; base < N; base += 4096) {
    const int64_t i0 = base + 4 * (int64_t)t;
    int32_t c[4];
    if (vec && i0 + 3 < N) {
      const i32x4 v = *reinterpret_cast<const i32x4*>(row_offsets + i0);
      c[0] = v[0], c[1] = v[1], c[2] = v[2], c[3] = v[3];
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = i0 + j < N ? row_offsets[i0 + j] : 0;
    }
    const int64_t s = (int64_t)c[0] + c[1] + c[2] + c[3];
    int64_t x = s;                                       // inclusive scan over the wave's threads
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int64_t y = __shfl_up(x, d);
      if (lane >= d) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int64_t before = carry + x - s, total = 0;
#pragma unroll
    for (int w = 0; w < 16; ++w) {
      const int64_t ws = wsum[w];
      if (w < wave) before += ws;
      total += ws;
    }
    int32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      o[j] = (int32_t)before;
      before += c[j];
    }
    if (vec && i0 + 3 < N) {
      *reinterpret_cast<i32x4*>(row_offsets + i0) = i32x4{o[0], o[1], o[2], o[3]};
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (i0 + j < N) row_offsets[i0 + j] = o[j];
    }
    carry += total;
    __syncthreads();                                     // wsum is rewritten by the next pass
  }
  if (t == 0) row_offsets[N] = carry >= (int64_t)2147483648LL ? -1 : (int32_t)carry;
}

template <int EB>
__global__ void __launch_bounds__(256) k_pack_scatter(const void* W, const uint8_t* mask, int64_t N, int64_t K,
                                                      const int32_t* row_offsets, uint32_t* bitmask,
                                                      void* values) {
  const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const uint32_t lane = threadIdx.x & 63u;
  const int64_t words = words_per_row(K);
  const int64_t base = n * K;
  uint32_t* brow = bitmask + n * words;
  int64_t out = row_offsets[n];
  for (int64_t k0 = 0; k0 < K; k0 += kWave) {
    const int64_t k = k0 + lane;
    const bool keep = k < K && is_kept<EB>(W, mask, base + k);
    const uint64_t b = __ballot(keep);
    if (keep) {
      const int64_t slot = out + mbcnt64(b);
      if constexpr (EB == 2) {
        static_cast<uint16_t*>(values)[slot] = static_cast<const uint16_t*>(W)[base + k];
      } else {
        static_cast<int8_t*>(values)[slot] = static_cast<const int8_t*>(W)[base + k];
      }
    }
    const int64_t w = k0 >> 5;
    if (lane == 0) brow[w] = (uint32_t)b;
    if (lane == 1 && w + 1 < words) brow[w + 1] = (uint32_t)(b >> 32);
    out += __popcll(b);
  }
}

template <int EB>
__global__ void __launch_bounds__(256) k_unpack(const uint32_t* bitmask, const void* values,
                                                const int32_t* row_offsets, int64_t N, int64_t K, void* Wd) {
  const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const uint32_t lane = threadIdx.x & 63u;
  const int64_t words = words_per_row(K);
  const uint32_t* brow = bitmask + n * words;
  int64_t in = row_offsets[n];
  for (int64_t k0 = 0; k0 < K; k0 += kWave) {
    const int64_t w = k0 >> 5;
    const uint64_t b = (uint64_t)brow[w] | (w + 1 < words ? (uint64_t)brow[w + 1] << 32 : 0ull);
    const int64_t k = k0 + lane;
    if (k < K) {
      const bool bit = (b >> lane) & 1ull;
      const int64_t src = in + mbcnt64(b);
      if constexpr (EB == 2) {
        static_cast<uint16_t*>(Wd)[n * K + k] = bit ? static_cast<const uint16_t*>(values)[src] : (uint16_t)0;
      } else {
        static_cast<int8_t*>(Wd)[n * K + k] = bit ? static_cast<const int8_t*>(values)[src] : (int8_t)0;
      }
    }
    in += __popcll(b);
  }
}

// ---- tile layout (16 x 32 submatrices) ----

// Thread (tile t, row r): copy the row's bitmask word into tile order and
// count the tile's kept entries into tile_offsets[t].
__global__ void __launch_bounds__(256) k_tile_count(const uint32_t* __restrict__ bm_rows, int64_t N, int64_t K,
                                                    uint32_t* __restrict__ bm_tiles, int32_t* __restrict__ counts) {
  const int64_t S = tile_steps(K);
  const int64_t T = tile_blocks(N) * S;
  const int64_t t = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int r = threadIdx.x & 15;
  uint32_t w = 0;
  if (t < T) {
    const int64_t b = t / S, s = t - b * S;
    const int64_t n = 16 * b + r;
    if (n < N) w = bm_rows[n * S + s];
    bm_tiles[t * 16 + r] = w;
  }
  uint32_t c = __popc(w);
  for (int off = 8; off > 0; off >>= 1) c += __shfl_xor(c, off, 16);
  if (t < T && r == 0) counts[t] = (int32_t)c;
}

// Position, inside tile t, of the first value of row r's column group g:
// tile values are ordered by column group (G columns = 16 bytes of payload),
// then row, then column, so it is the kept count of every row below group g
// plus that of the rows above r inside group g.  `words` holds the tile's 16
// bitmask words.
template <int G>
__device__ __forceinline__ uint32_t tile_group_start(const uint32_t (&words)[16], int r, int g) {
  const uint32_t below = (1u << (G * g)) - 1u;                           // G g < 32
  const uint32_t gm = (G == 32 ? 0xffffffffu : ((1u << G) - 1u)) << (G * g);
  uint32_t pos = 0;
#pragma unroll
  for (int rr = 0; rr < 16; ++rr) pos += __popc(words[rr] & below) + (rr < r ? __popc(words[rr] & gm) : 0u);
  return pos;
}

// One wave per row: for each 32-column word, the row's stored values move from
// their row-layout position to their tile-layout position, group by group.
template <int EB>
__global__ void __launch_bounds__(256) k_tile_scatter(const uint32_t* __restrict__ bm_rows,
                                                      const void* __restrict__ vals_rows,
                                                      const int32_t* __restrict__ row_offsets, int64_t N, int64_t K,
                                                      const int32_t* __restrict__ tile_offsets,
                                                      void* __restrict__ vals_tiles) {
  constexpr int G = 16 / EB;                           // columns per group
  const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const int lane = threadIdx.x & 63;
  const int64_t S = tile_steps(K);
  const int64_t b = n / 16;
  const int r = (int)(n - 16 * b);
  int64_t carry = row_offsets[n];
  for (int64_t s0 = 0; s0 < S; s0 += kWave) {
    const int64_t s = s0 + lane;
    const uint32_t w = s < S ? bm_rows[n * S + s] : 0u;
    const uint32_t pc = __popc(w);
    uint32_t incl = pc;
    for (int d = 1; d < kWave; d <<= 1) {
      const uint32_t up = __shfl_up(incl, d);
      if (lane >= d) incl += up;
    }
    const uint32_t total = __shfl(incl, kWave - 1);
    if (pc) {
      uint32_t words[16];
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) words[rr] = 16 * b + rr < N ? bm_rows[(16 * b + rr) * S + s] : 0u;
      int64_t src = carry + (incl - pc);
      const int64_t t0 = tile_offsets[b * S + s];
#pragma unroll
      for (int g = 0; g < 32 / G; ++g) {
        const uint32_t cg = __popc(w & (((1u << G) - 1u) << (G * g)));
        const int64_t dst = t0 + tile_group_start<G>(words, r, g);
        for (uint32_t i = 0; i < cg; ++i) {
          if constexpr (EB == 2) {
            static_cast<uint16_t*>(vals_tiles)[dst + i] = static_cast<const uint16_t*>(vals_rows)[src + i];
          } else {
            static_cast<int8_t*>(vals_tiles)[dst + i] = static_cast<const int8_t*>(vals_rows)[src + i];
          }
        }
        src += cg;
      }
    }
    carry += total;
  }
}

// The dense image of a 16-bit tile-layout matrix with K % 8 == 0.  A wave
// expands kExpandTiles consecutive tiles (4 per workgroup of 4 waves), with
// every tile's loads in flight together: lane (fr, fg) writes row fr, columns
// 8 fg .. 8 fg + 7 of each with one 16-byte store.  A tile's values are in
// lane order, so the lane's first value is the tile offset + the exclusive
// wave scan of the lanes' kept counts (two tiles per scan, in 16-bit halves);
// two 8-byte windows from the first value of each of its nibbles are expanded
// by a 16-entry selector table with v_perm_b32 (zero where a bit is clear).
// A window reads at most 3 values past the last kept one: inside the 16
// readable bytes that follow the payload.
constexpr int kExpandTiles = 4;
__global__ void __launch_bounds__(256) k_expand_tiles16(const uint32_t* __restrict__ bm_tiles,
                                                        const uint16_t* __restrict__ values,
                                                        const int32_t* __restrict__ tile_offsets, int64_t N,
                                                        int64_t K, int64_t tiles, uint16_t* __restrict__ Wd) {
  __shared__ u32x2 lut[16];
  if (threadIdx.x < 16) lut[threadIdx.x] = u32x2{nibble_selector16(threadIdx.x, 0), nibble_selector16(threadIdx.x, 1)};
  __syncthreads();
  const int64_t t0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * kExpandTiles;
  if (t0 >= tiles) return;                           // whole waves leave together
  const int lane = threadIdx.x & 63, fr = lane & 15, fg = lane >> 4;
  const int64_t S = tile_steps(K);
  uint32_t byte[kExpandTiles], oa[kExpandTiles];
#pragma unroll
  for (int i = 0; i < kExpandTiles; ++i) {          // tiles past the end: no kept bits, no store
    const bool live = t0 + i < tiles;
    byte[i] = live ? (bm_tiles[(t0 + i) * 16 + fr] >> (8 * fg)) & 0xffu : 0u;   // pad rows, columns: 0
    oa[i] = live ? (uint32_t)tile_offsets[t0 + i] : 0u;
  }
#pragma unroll
  for (int i = 0; i < kExpandTiles; i += 2) {
    const uint32_t pc = __popc(byte[i]) | (__popc(byte[i + 1]) << 16);
    const uint32_t ex = wave_inclusive_scan(pc) - pc;
    oa[i] += ex & 0xffffu;
    oa[i + 1] += ex >> 16;
  }
  u32x2 v0[kExpandTiles], v1[kExpandTiles];
#pragma unroll
  for (int i = 0; i < kExpandTiles; ++i) {
    if (byte[i] != 0u) {
      __builtin_memcpy(&v0[i], values + oa[i], 8);
      __builtin_memcpy(&v1[i], values + oa[i] + __popc(byte[i] & 0xfu), 8);
    }
  }
#pragma unroll
  for (int i = 0; i < kExpandTiles; ++i) {
    const int64_t t = t0 + i;
    const int64_t n = (t / S) * 16 + fr;
    const int64_t k0 = (t % S) * 32 + 8 * fg;
    if (t >= tiles || n >= N || k0 >= K) continue;
    u32x4 a = u32x4{0u, 0u, 0u, 0u};
    if (byte[i] != 0u) {
      const u32x2 slo = lut[byte[i] & 0xfu], shi = lut[byte[i] >> 4];
      a.x = __builtin_amdgcn_perm(v0[i].y, v0[i].x, slo.x);
      a.y = __builtin_amdgcn_perm(v0[i].y, v0[i].x, slo.y);
      a.z = __builtin_amdgcn_perm(v1[i].y, v1[i].x, shi.x);
      a.w = __builtin_amdgcn_perm(v1[i].y, v1[i].x, shi.y);
    }
    *reinterpret_cast<u32x4*>(Wd + n * K + k0) = a;  // K % 8 == 0 and Wd 16-byte aligned
  }
}

// The same for an int8 tile-layout matrix with K % 16 == 0: a wave expands
// 2 kExpandTiles consecutive tiles, tile pair p being tiles 2p (lanes 0-31)
// and 2p + 1 (lanes 32-63); lane (r, g) of a tile (r = lane % 16, g = lane /
// 16 % 2) writes row r, columns 16 g .. 16 g + 15 with one 16-byte store.  A
// tile's int8 values are ordered by 16-column group, then row (the order of
// its 32 lanes), so the lane's first value is the tile offset + the exclusive
// scan over its half-wave of the lanes' kept counts; the 8-byte windows from
// the first value of columns 0-7 and of columns 8-15 of its group are
// expanded per nibble by a selector table indexed by the nibble and the place
// of its first value in the window.  A window reads at most 7 bytes past the
// last kept value: inside the 16 readable bytes that follow the payload.
__global__ void __launch_bounds__(256) k_expand_tiles8(const uint32_t* __restrict__ bm_tiles,
                                                       const uint8_t* __restrict__ values,
                                                       const int32_t* __restrict__ tile_offsets, int64_t N,
                                                       int64_t K, int64_t tiles, uint8_t* __restrict__ Wd) {
  __shared__ uint32_t lut[80];
  if (threadIdx.x < 80) lut[threadIdx.x] = nibble_selector8(threadIdx.x / 5, threadIdx.x % 5);
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t t0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * 2 * kExpandTiles;
  if (t0 >= tiles) return;                           // whole waves leave together
  const int r = lane & 15, gq = (lane >> 4) & 1;
  const int64_t S = tile_steps(K);
  uint32_t hw[kExpandTiles], oa[kExpandTiles];
#pragma unroll
  for (int p = 0; p < kExpandTiles; ++p) {
    const int64_t t = t0 + 2 * p + (lane >> 5);
    const bool live = t < tiles;
    hw[p] = live ? (bm_tiles[t * 16 + r] >> (16 * gq)) & 0xffffu : 0u;   // pad rows, columns: 0
    oa[p] = live ? (uint32_t)tile_offsets[t] : 0u;
  }
#pragma unroll
  for (int p = 0; p < kExpandTiles; p += 2) {
    const uint32_t pc = __popc(hw[p]) | (__popc(hw[p + 1]) << 16);
    const uint32_t ex = half_inclusive_scan(pc) - pc;
    oa[p] += ex & 0xffffu;
    oa[p + 1] += ex >> 16;
  }
  u32x2 v0[kExpandTiles], v1[kExpandTiles];
#pragma unroll
  for (int p = 0; p < kExpandTiles; ++p) {
    if (hw[p] != 0u) {
      __builtin_memcpy(&v0[p], values + oa[p], 8);
      __builtin_memcpy(&v1[p], values + oa[p] + __popc(hw[p] & 0xffu), 8);   // columns 8-15 after 0-7
    }
  }
#pragma unroll
  for (int p = 0; p < kExpandTiles; ++p) {
    const int64_t t = t0 + 2 * p + (lane >> 5);
    const int64_t n = (t / S) * 16 + r;
    const int64_t k0 = (t % S) * 32 + 16 * gq;
    if (t >= tiles || n >= N || k0 >= K) continue;
    u32x4 a = u32x4{0u, 0u, 0u, 0u};
    if (hw[p] != 0u) {
      const uint32_t q0 = hw[p] & 15u, q1 = (hw[p] >> 4) & 15u, q2 = (hw[p] >> 8) & 15u, q3 = hw[p] >> 12;
      a.x = __builtin_amdgcn_perm(v0[p].y, v0[p].x, lut[5 * q0]);
      a.y = __builtin_amdgcn_perm(v0[p].y, v0[p].x, lut[5 * q1 + __popc(q0)]);
      a.z = __builtin_amdgcn_perm(v1[p].y, v1[p].x, lut[5 * q2]);
      a.w = __builtin_amdgcn_perm(v1[p].y, v1[p].x, lut[5 * q3 + __popc(q2)]);
    }
    *reinterpret_cast<u32x4*>(Wd + n * K + k0) = a;  // K % 16 == 0 and Wd 16-byte aligned
  }
}

// Thread (tile t, row r): decode one tile row into the dense matrix.
template <int EB>
__global__ void __launch_bounds__(256) k_unpack_tiled(const uint32_t* __restrict__ bm_tiles,
                                                      const void* __restrict__ values,
                                                      const int32_t* __restrict__ tile_offsets, int64_t N, int64_t K,
                                                      void* __restrict__ Wd) {
  constexpr int G = 16 / EB;
  const int64_t S = tile_steps(K);
  const int64_t T = tile_blocks(N) * S;
  const int64_t t = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int r = threadIdx.x & 15;
  if (t >= T) return;
  const int64_t b = t / S, s = t - b * S;
  const int64_t n = 16 * b + r;
  if (n >= N) return;
  uint32_t words[16];
#pragma unroll
  for (int rr = 0; rr < 16; ++rr) words[rr] = bm_tiles[t * 16 + rr];
  const uint32_t w = words[r];
  for (int g = 0; g < 32 / G; ++g) {
    int64_t src = tile_offsets[t] + tile_group_start<G>(words, r, g);
    for (int j = G * g; j < G * g + G; ++j) {
      const int64_t k = 32 * s + j;
      if (k >= K) break;
      const bool bit = (w >> j) & 1u;
      if constexpr (EB == 2) {
        static_cast<uint16_t*>(Wd)[n * K + k] = bit ? static_cast<const uint16_t*>(values)[src] : (uint16_t)0;
      } else {
        static_cast<int8_t*>(Wd)[n * K + k] = bit ? static_cast<const int8_t*>(values)[src] : (int8_t)0;
      }
      src += bit;
    }
  }
}


// ---- pack straight into the tile layout ----

// Thread (tile t, row r): the kept count of its 32 columns, summed per tile.
template <int EB>
__global__ void __launch_bounds__(256) k_tile_count_direct(const void* W, const uint8_t* mask, int64_t N, int64_t K,
                                                           int32_t* __restrict__ counts) {
  const int64_t S = tile_steps(K);
  const int64_t T = tile_blocks(N) * S;
  const int64_t t = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int r = threadIdx.x & 15;
  uint32_t c = 0;
  if (t < T) {
    const int64_t b = t / S, s = t - b * S;
    const int64_t n = 16 * b + r;
    if (n < N) {
      const int64_t k0 = 32 * s;
      const int64_t k1 = k0 + 32 < K ? k0 + 32 : K;
      for (int64_t k = k0; k < k1; ++k) c += is_kept<EB>(W, mask, n * K + k) ? 1u : 0u;
    }
  }
  for (int off = 8; off > 0; off >>= 1) c += __shfl_xor(c, off, 16);
  if (t < T && r == 0) counts[t] = (int32_t)c;
}

// One wave per tile.  Lane (fr, g) covers row fr and the G = 16 / EB columns
// of group g (EB = 2: 64 lanes, 4 groups of 8; EB = 1: 32 lanes, 2 groups of
// 16), which is the order of the tile's values, so the lane's first value sits
// at the exclusive scan of the lanes' counts.  It writes its kept values in
// column order and its G bits of the row's bitmask word (byte g, or half-word
// g for int8), zero for rows >= N and columns >= K.
template <int EB>
__global__ void __launch_bounds__(256) k_tile_scatter_direct(const void* W, const uint8_t* mask, int64_t N,
                                                             int64_t K, const int32_t* __restrict__ tile_offsets,
                                                             uint32_t* __restrict__ bm_tiles, void* __restrict__ values) {
  constexpr int G = 16 / EB;
  constexpr int kLanes = 16 * (32 / G);
  const int64_t S = tile_steps(K);
  const int64_t T = tile_blocks(N) * S;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;                                    // wave-uniform
  const int lane = threadIdx.x & 63;
  const int fr = lane & 15, g = lane >> 4;
  const int64_t b = t / S, s = t - b * S;
  const int64_t n = 16 * b + fr;
  const int64_t k0 = 32 * s + (int64_t)G * g;
  uint32_t bits = 0;
  if (lane < kLanes && n < N) {
#pragma unroll
    for (int j = 0; j < G; ++j)
      if (k0 + j < K && is_kept<EB>(W, mask, n * K + k0 + j)) bits |= 1u << j;
  }
  const uint32_t c = __popc(bits);
  uint32_t incl = c;
  for (int d = 1; d < kWave; d <<= 1) {
    const uint32_t up = __shfl_up(incl, d);
    if (lane >= d) incl += up;
  }
  int64_t dst = (int64_t)tile_offsets[t] + (incl - c);
  if (lane < kLanes) {
    unsigned char* wb = reinterpret_cast<unsigned char*>(bm_tiles + t * 16 + fr);
    if constexpr (EB == 2) {
      wb[g] = (unsigned char)bits;
    } else {
      *reinterpret_cast<uint16_t*>(wb + 2 * g) = (uint16_t)bits;
    }
    for (int j = 0; j < G; ++j) {
      if ((bits >> j) & 1u) {
        if constexpr (EB == 2) {
          static_cast<uint16_t*>(values)[dst] = static_cast<const uint16_t*>(W)[n * K + k0 + j];
        } else {
          static_cast<int8_t*>(values)[dst] = static_cast<const int8_t*>(W)[n * K + k0 + j];
        }
        ++dst;
      }
    }
  }
}

// ---- format check ----

// Error bits of spl_validate.
constexpr uint32_t kBadCount = 1u;     // offsets[i+1] - offsets[i] != kept count of block i
constexpr uint32_t kBadEnds = 2u;      // offsets[0] != 0 or offsets[last] != nnz
constexpr uint32_t kBadPad = 4u;       // a bit set past column K or (tile layout) in a row >= N

// Thread per block (a row, or a tile): its popcount against its offsets, its pad bits.
__global__ void __launch_bounds__(256) k_validate(const uint32_t* __restrict__ bitmask,
                                                  const int32_t* __restrict__ offsets, int64_t N, int64_t K,
                                                  int64_t nnz, int tiled, uint32_t* __restrict__ err) {
  const int64_t S = tile_steps(K);
  const int64_t blocks = tiled ? tile_blocks(N) * S : N;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i > blocks) return;
  uint32_t e = 0;
  if (i == blocks) {
    if (offsets[0] != 0 || (int64_t)offsets[blocks] != nnz) e |= kBadEnds;
  } else {
    const uint32_t tail = (uint32_t)(K - 32 * (S - 1));                  // columns of the last 32-column step
    const uint32_t tailmask = tail >= 32 ? 0xffffffffu : ((1u << tail) - 1u);
    int64_t c = 0;
    if (tiled) {
      const int64_t b = i / S, s = i - b * S;
#pragma unroll 4
      for (int r = 0; r < 16; ++r) {
        const uint32_t w = bitmask[i * 16 + r];
        c += __popc(w);
        if ((16 * b + r >= N && w) || (s == S - 1 && (w & ~tailmask))) e |= kBadPad;
      }
    } else {
      for (int64_t s = 0; s < S; ++s) {
        const uint32_t w = bitmask[i * S + s];
        c += __popc(w);
        if (s == S - 1 && (w & ~tailmask)) e |= kBadPad;
      }
    }
    if ((int64_t)offsets[i + 1] - (int64_t)offsets[i] != c) e |= kBadCount;
  }
  if (e) atomicOr(err, e);
}

__global__ void k_clear_word(uint32_t* w) { *w = 0u; }

}  // namespace

hipError_t launch_retile16(const spl_matrix& in, uint32_t* bitmask_t, void* values_t, int32_t* tile_offsets,
                           hipStream_t s) {
  const int64_t T = tile_blocks(in.rows) * tile_steps(in.cols);
  hipLaunchKernelGGL(k_tile_count, dim3((unsigned)((T + 15) / 16)), dim3(256), 0, s, in.bitmask, in.rows, in.cols,
                     bitmask_t, tile_offsets);
  hipLaunchKernelGGL(k_scan_offsets, dim3(1), dim3(1024), 0, s, tile_offsets, T);
  if (in.nnz > 0) {
    const dim3 grid((unsigned)((in.rows + 3) / 4)), block(256);
    if (in.dtype == SPL_I8) {
      hipLaunchKernelGGL(k_tile_scatter<1>, grid, block, 0, s, in.bitmask, in.values, in.row_offsets, in.rows,
                         in.cols, tile_offsets, values_t);
    } else {
      hipLaunchKernelGGL(k_tile_scatter<2>, grid, block, 0, s, in.bitmask, in.values, in.row_offsets, in.rows,
                         in.cols, tile_offsets, values_t);
    }
  }
  return hipGetLastError();
}

hipError_t launch_pack_count(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
                             int32_t* row_offsets, hipStream_t s) {
  const dim3 grid((unsigned)((N + 3) / 4)), block(256);
  if (dtype == SPL_I8) {
    hipLaunchKernelGGL(k_row_count<1>, grid, block, 0, s, W, mask, N, K, row_offsets);
  } else {
    hipLaunchKernelGGL(k_row_count<2>, grid, block, 0, s, W, mask, N, K, row_offsets);
  }
  hipLaunchKernelGGL(k_scan_offsets, dim3(1), dim3(1024), 0, s, row_offsets, N);
  return hipGetLastError();
}

hipError_t launch_pack_scatter(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
                               const int32_t* row_offsets, uint32_t* bitmask, void* values, hipStream_t s) {
  const dim3 grid((unsigned)((N + 3) / 4)), block(256);
  if (dtype == SPL_I8) {
    hipLaunchKernelGGL(k_pack_scatter<1>, grid, block, 0, s, W, mask, N, K, row_offsets, bitmask, values);
  } else {
    hipLaunchKernelGGL(k_pack_scatter<2>, grid, block, 0, s, W, mask, N, K, row_offsets, bitmask, values);
  }
  return hipGetLastError();
}

hipError_t launch_pack_count_tiled(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
                                   int32_t* tile_offsets, hipStream_t s) {
  const int64_t T = tile_blocks(N) * tile_steps(K);
  const dim3 grid((unsigned)((T + 15) / 16)), block(256);
  if (dtype == SPL_I8) {
    hipLaunchKernelGGL(k_tile_count_direct<1>, grid, block, 0, s, W, mask, N, K, tile_offsets);
  } else {
    hipLaunchKernelGGL(k_tile_count_direct<2>, grid, block, 0, s, W, mask, N, K, tile_offsets);
  }
  hipLaunchKernelGGL(k_scan_offsets, dim3(1), dim3(1024), 0, s, tile_offsets, T);
  return hipGetLastError();
}

hipError_t launch_pack_scatter_tiled(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
                                     const int32_t* tile_offsets, uint32_t* bitmask, void* values, hipStream_t s) {
  const int64_t T = tile_blocks(N) * tile_steps(K);
  const dim3 grid((unsigned)((T + 3) / 4)), block(256);
  if (dtype == SPL_I8) {
    hipLaunchKernelGGL(k_tile_scatter_direct<1>, grid, block, 0, s, W, mask, N, K, tile_offsets, bitmask, values);
  } else {
    hipLaunchKernelGGL(k_tile_scatter_direct<2>, grid, block, 0, s, W, mask, N, K, tile_offsets, bitmask, values);
  }
  return hipGetLastError();
}

hipError_t launch_validate(const spl_matrix& Wc, uint32_t* err, hipStream_t s) {
  hipLaunchKernelGGL(k_clear_word, dim3(1), dim3(1), 0, s, err);
  const bool tiled = Wc.layout == SPL_LAYOUT_TILE16;
  const int64_t blocks = tiled ? tile_blocks(Wc.rows) * tile_steps(Wc.cols) : Wc.rows;
  hipLaunchKernelGGL(k_validate, dim3((unsigned)((blocks + 1 + 255) / 256)), dim3(256), 0, s, Wc.bitmask,
                     tiled ? Wc.tile_offsets : Wc.row_offsets, Wc.rows, Wc.cols, Wc.nnz, tiled ? 1 : 0, err);
  return hipGetLastError();
}

hipError_t launch_unpack(const spl_matrix& Wc, void* W_dense, hipStream_t s) {
  if (Wc.layout == SPL_LAYOUT_TILE16) {
    const int64_t T = tile_blocks(Wc.rows) * tile_steps(Wc.cols);
    if (Wc.dtype != SPL_I8 && Wc.cols % 8 == 0) {   // W_dense is 16-byte aligned (checked by the caller)
      hipLaunchKernelGGL(k_expand_tiles16, dim3((unsigned)((T + 4 * kExpandTiles - 1) / (4 * kExpandTiles))),
                         dim3(256), 0, s, Wc.bitmask,
                         static_cast<const uint16_t*>(Wc.values), Wc.tile_offsets, Wc.rows, Wc.cols, T,
                         static_cast<uint16_t*>(W_dense));
      return hipGetLastError();
    }
    if (Wc.dtype == SPL_I8 && Wc.cols % 16 == 0) {
      hipLaunchKernelGGL(k_expand_tiles8, dim3((unsigned)((T + 8 * kExpandTiles - 1) / (8 * kExpandTiles))),
                         dim3(256), 0, s, Wc.bitmask,
                         static_cast<const uint8_t*>(Wc.values), Wc.tile_offsets, Wc.rows, Wc.cols, T,
                         static_cast<uint8_t*>(W_dense));
      return hipGetLastError();
    }
    const dim3 grid((unsigned)((T + 15) / 16)), block(256);
    if (Wc.dtype == SPL_I8) {
      hipLaunchKernelGGL(k_unpack_tiled<1>, grid, block, 0, s, Wc.bitmask, Wc.values, Wc.tile_offsets, Wc.rows,
                         Wc.cols, W_dense);
    } else {
      hipLaunchKernelGGL(k_unpack_tiled<2>, grid, block, 0, s, Wc.bitmask, Wc.values, Wc.tile_offsets, Wc.rows,
                         Wc.cols, W_dense);
    }
    return hipGetLastError();
  }
  const dim3 grid((unsigned)((Wc.rows + 3) / 4)), block(256);
  if (Wc.dtype == SPL_I8) {
    hipLaunchKernelGGL(k_unpack<1>, grid, block, 0, s, Wc.bitmask, Wc.values, Wc.row_offsets, Wc.rows, Wc.cols,
                       W_dense);
  } else {
    hipLaunchKernelGGL(k_unpack<2>, grid, block, 0, s, Wc.bitmask, Wc.values, Wc.row_offsets, Wc.rows, Wc.cols,
                       W_dense);
  }
  return hipGetLastError();
}

}  // namespace spl
