// Sparse-quantized linear layer (paper section 3.4: int8 weights and int8
// activations) and its dense comparator, for gfx950.
//
// acc[m][n] = sum over kept k of Xq[m][k] * Wq[n][k] is accumulated exactly in
// int32 by v_mfma_i32_16x16x64_i8; the epilogue is
//   Y[m][n] = fp16_rne( (float(acc) * sx[m]) * sw[n] )
// with each product rounded to binary32 (no fused multiply-add).
//
// Sparse kernel (the decode kernel's design with 1-byte payloads): a
// workgroup owns one 16-row block and its waves split the block's tile pairs
// into contiguous ranges.  One MFMA covers a pair of consecutive 16 x 32
// tiles: lanes 0-31 take tile s, lanes 32-63 tile s + 1, lane (fr, fg) row fr,
// columns 16 (fg % 2) .. +16 of its tile.  A wave stages a chunk of tiles
// (whole pairs, as many as fit a 3 KB buffer) with aligned 16-byte loads in
// LDS, the tile offsets of its whole range come with one load, and the next
// chunk is in flight while the current one is multiplied.  Each lane expands
// its four 4-column nibbles: a tile's values are stored by 16-column group,
// then row, i.e. in the order of the tile's 32 lanes, so the nibble's values
// start at the tile offset + the kept count of the lanes before (a 32-lane
// DPP scan) + the nibbles before it, are read as an aligned dword pair realigned with
// v_alignbyte_b32, and a 16-entry selector table (conflict-free) drives
// v_perm_b32 (paper section 2.4.1).  Activations of small batches are staged
// in LDS once per workgroup; int32 partial sums of the waves are added in LDS
// (integer addition: the order does not matter).
#include "spl_common.h"

namespace spl {
namespace {

constexpr int kI8Waves = 8;                 // dense kernel
constexpr int kI8Threads = 64 * kI8Waves;
constexpr int kI8Unroll = 4;                // dense kernel: 64-column steps per wave per group
constexpr int kI8Chunk = 8;                 // sparse: at most this many tiles (4 pairs) per chunk (4 when M > 32)
constexpr int kI8VBuf = 3072;               // staged value bytes per wave and chunk
constexpr int kI8VBufAlloc = kI8VBuf + 16;  // + room past the last window
constexpr int kI8PieceRounds = kI8VBuf / 16 / kWave;
constexpr int kI8XLdsMax = 32 * 1024;       // activations staged in LDS when M * 64 ceil(S/2) bytes fit
constexpr int kI8OffsetLanes = kWave - 1;
// Batches from this size on use the prefill kernels' MFMA tiling (activations staged in LDS and
// shared by the row blocks of a workgroup) instead of the streaming kernels below.
constexpr int64_t kI8PrefillMinM = 128;

__device__ __forceinline__ i32x4 mfma_i8(u32x4 a, u32x4 b, i32x4 c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, a), __builtin_bit_cast(i32x4, b), c, 0, 0,
                                               0);
}

// Combine the waves' int32 partial sums and run the epilogue.
// part: [W][MT][4][64] int32 in LDS; output (f, r, l): n = n0 + 4*(l/16) + r, m = m0 + 16 f + l%16.
template <int MT, int W>
__device__ __forceinline__ void i8_finish(const i32x4 (&acc)[MT], int32_t* part, int wave, int lane, int64_t n0,
                                          int64_t N, int64_t m0, int64_t M, const float* __restrict__ sx,
                                          const float* __restrict__ sw, uint16_t* __restrict__ Y,
                                          int32_t* __restrict__ acc_out) {
#pragma unroll
  for (int f = 0; f < MT; ++f)
#pragma unroll
    for (int r = 0; r < 4; ++r) part[((wave * MT + f) * 4 + r) * 64 + lane] = acc[f][r];
  __syncthreads();
  for (int o = threadIdx.x; o < MT * 4 * 64; o += W * kWave) {
    const int f = o / 256, r = (o / 64) & 3, l = o & 63;
    const int64_t n = n0 + 4 * (l >> 4) + r;
    const int64_t m = m0 + 16 * f + (l & 15);
    if (n < N && m < M) {
      int32_t s = 0;
#pragma unroll
      for (int w = 0; w < W; ++w) s += part[w * MT * 256 + o];
      if (acc_out) acc_out[m * N + n] = s;
      const float a = static_cast<float>(s);
      const float t = __fmul_rn(a, sx[m]);
      const float y = __fmul_rn(t, sw[n]);
      Y[m * N + n] = F16::from_f32(y);
    }
  }
}

// int8 activations staged in LDS: rows of 64 * ceil(S / 2) + 16 bytes (whole
// tile pairs, so the second tile of a last half pair reads zeros), zero past
// K.  Lanes of padding batch rows read a 64-byte zero area and do not advance.
__host__ __device__ __forceinline__ int64_t i8_xs_stride(int64_t K) { return 64 * ((tile_steps(K) + 1) / 2) + 16; }

template <int W>
__device__ __forceinline__ void i8_stage_x(uint8_t* xs, const int8_t* __restrict__ X, int M, int64_t K) {
  const int per_row = (int)(4 * ((tile_steps(K) + 1) / 2));   // 16-byte pieces per staged row (whole pairs)
  const int kp = (int)(K / 16);                           // pieces holding activations
  const int total = M * per_row;
  for (int p = threadIdx.x; p < total; p += W * kWave) {
    const int m = p / per_row, q = p - m * per_row;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (q < kp) v = *reinterpret_cast<const u32x4*>(X + (int64_t)m * K + 16 * q);
    *reinterpret_cast<u32x4*>(xs + (int64_t)m * i8_xs_stride(K) + 16 * q) = v;
  }
}

struct I8Chunk {
  int cn;
  uint32_t a0;
  int np;
};

// Grouped launches: task i owns the row blocks [first[i], first[i + 1]) of the
// grid's x dimension; every task has the group's batch M (grid y).
struct I8TaskArg {
  const int8_t* Xq;
  const float* sx;
  const uint32_t* bm;
  const uint8_t* values;
  const int32_t* toff;
  int64_t N, K;
  const float* sw;
  uint16_t* Y;
  int32_t* acc;
};
struct I8GroupArg {
  I8TaskArg t[SPL_MAX_GROUP];
  int32_t first[SPL_MAX_GROUP + 1];
  int32_t count;
  int32_t M;
};
struct I8DenseTaskArg {
  const int8_t* Xq;
  const float* sx;
  const int8_t* W;
  int64_t N, K;
  const float* sw;
  uint16_t* Y;
  int32_t* acc;
};
struct I8DenseGroupArg {
  I8DenseTaskArg t[SPL_MAX_GROUP];
  int32_t first[SPL_MAX_GROUP + 1];
  int32_t count;
  int32_t M;
};

template <int MT, bool XL, int W>
__global__ void __launch_bounds__(W * kWave, XL ? 8 : 4) k_sparse_int8(const I8GroupArg g) {
  const int ti = find_task(g.first, g.count);
  const I8TaskArg tk = g.t[ti];
  const int8_t* __restrict__ Xq = tk.Xq;
  const float* __restrict__ sx = tk.sx;
  const int64_t M = g.M, K = tk.K, N = tk.N;
  const uint32_t* __restrict__ bm_tiles = tk.bm;
  const uint8_t* __restrict__ values = tk.values;
  const int32_t* __restrict__ tile_offsets = tk.toff;
  const float* __restrict__ sw = tk.sw;
  uint16_t* __restrict__ Y = tk.Y;
  int32_t* __restrict__ acc_out = tk.acc;
  constexpr int C = MT == 4 ? kI8Chunk / 2 : kI8Chunk;     // four batch fragments: half the operands in flight
  extern __shared__ __align__(16) unsigned char dsm[];     // value buffers (later the partial sums), then X
  __shared__ uint32_t lut[16];
  __shared__ u32x4 xzero[4];
  // per wave: [row][tile of the chunk]; the odd row stride C + 1 puts the 16 rows in distinct banks
  constexpr int WS = C + 1;
  __shared__ __align__(16) uint32_t words[W][16 * WS];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int fr = lane & 15, fg = lane >> 4;
  const int tsel = fg >> 1, half = fg & 1;
  const int64_t blk = (int64_t)blockIdx.x - g.first[ti];
  const int64_t m0 = (int64_t)blockIdx.y * 16 * MT;
  const int S = (int)tile_steps(K);
  const int P = (S + 1) / 2;
  // this wave's tiles: whole pairs [2 pb, 2 pe) clipped to S
  int kbeg, kend;
  {
    const int Lp = (P + W - 1) / W;
    const int pb = wave * Lp < P ? wave * Lp : P;
    const int pe = pb + Lp < P ? pb + Lp : P;
    kbeg = 2 * pb;
    kend = 2 * pe < S ? 2 * pe : S;
    if (kbeg > kend) kbeg = kend;
  }
  const size_t vbytes_region = (size_t)W * kI8VBufAlloc > (size_t)W * MT * 1024 ? (size_t)W * kI8VBufAlloc
                                                                                  : (size_t)W * MT * 1024;
  unsigned char* vbuf = dsm + wave * kI8VBufAlloc;
  uint8_t* xs = reinterpret_cast<uint8_t*>(dsm + vbytes_region);
  const uint32_t* bmb = bm_tiles + blk * S * 16;
  const int32_t* tob = tile_offsets + blk * S;
  uint32_t* wl = words[wave];

  int ob = kbeg;
  auto load_offsets = [&](int base) {
    const int t = base + lane < kend ? base + lane : kend;
    return tob[t];
  };
  // whole pairs that fit the staging buffer (1-byte values: offsets are byte positions)
  auto shape = [&](int32_t o, int c0) {
    I8Chunk ch;
    const int r = c0 - ob;
    ch.a0 = (uint32_t)__builtin_amdgcn_readlane(o, r) & ~15u;
    const uint32_t lim = ch.a0 + kI8VBuf;
    const int jmax = kend - c0 < C ? kend - c0 : C;
    const bool fit = lane >= r + 1 && lane <= r + jmax && (uint32_t)o <= lim;
    int cn = __builtin_popcountll(__ballot(fit));          // >= 2 when jmax >= 2: two tiles are at most 1 KB
    if (cn < jmax) cn &= ~1;                                // chunks end on a pair boundary, or at the range end
    ch.cn = cn;
    const uint32_t end = (uint32_t)__builtin_amdgcn_readlane(o, r + cn);
    ch.np = (int)((end - ch.a0 + 15u) >> 4);
    return ch;
  };
  u32x4 vp[kI8PieceRounds];
  uint32_t wv[C / 4];
  auto issue = [&](const I8Chunk& ch, int c0) {
#pragma unroll
    for (int r = 0; r < kI8PieceRounds; ++r) {
      vp[r] = u32x4{0u, 0u, 0u, 0u};
      const uint32_t off = ch.a0 + 16u * (uint32_t)(lane + kWave * r);
      if (lane + kWave * r < ch.np) vp[r] = *reinterpret_cast<const u32x4*>(values + off);
    }
#pragma unroll
    for (int i = 0; i < C / 4; ++i) {
      wv[i] = 0u;
      const uint32_t wi = (uint32_t)(c0 + fg + 4 * i) * 16u + (uint32_t)fr;
      if (fg + 4 * i < ch.cn) wv[i] = bmb[wi];
    }
  };

  int32_t orng = 0;
  I8Chunk ch{0, 0u, 0};
  if (kbeg < kend) {
    orng = load_offsets(ob);
    ch = shape(orng, kbeg);
    issue(ch, kbeg);
  }
  if (threadIdx.x < 16) lut[threadIdx.x] = nibble_selector8(threadIdx.x);
  if (threadIdx.x < 4) xzero[threadIdx.x] = u32x4{0u, 0u, 0u, 0u};
  if constexpr (XL) i8_stage_x<W>(xs, Xq, (int)M, K);
  __syncthreads();

  // activation operands: staged (XL) or direct
  uint32_t xaddr0 = 0, xstep = 0;
  if constexpr (XL) {
    const bool live = fr < M;
    xaddr0 = live ? lds_off(xs + (int64_t)fr * i8_xs_stride(K) + 16 * fg) : lds_off(xzero + fg);
    xstep = live ? 64u : 0u;
  }
  const int8_t* xrow[MT];
  bool xlive[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int64_t m = m0 + 16 * t + fr;
    xlive[t] = m < M;
    xrow[t] = Xq + (xlive[t] ? m : 0) * K + 16 * fg;
  }
  const uint32_t lut_addr = lds_off(lut);
  const uint32_t vbuf_addr = lds_off(vbuf);
  u32x4 xs_op = u32x4{0u, 0u, 0u, 0u};

  i32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = i32x4{0, 0, 0, 0};

  for (int c0 = kbeg; c0 < kend;) {
    // 1. stage the current chunk
#pragma unroll
    for (int r = 0; r < kI8PieceRounds; ++r)
      if (lane + kWave * r < ch.np) *reinterpret_cast<u32x4*>(vbuf + 16 * (lane + kWave * r)) = vp[r];
#pragma unroll
    for (int i = 0; i < C / 4; ++i) wl[fr * WS + fg + 4 * i] = wv[i];
    wave_lds_sync();
    const I8Chunk cur = ch;
    int32_t tc[C];
#pragma unroll
    for (int j = 0; j < C; ++j) tc[j] = __builtin_amdgcn_readlane(orng, c0 - ob + j);

    // 2. direct activations for this chunk, then the next chunk's loads
    u32x4 xb[XL ? 1 : C / 2][MT];
    if constexpr (!XL) {
#pragma unroll
      for (int q = 0; q < C / 2; ++q)
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          const int64_t k = 32 * (int64_t)(c0 + 2 * q) + 16 * fg;
          xb[q][t] = u32x4{0u, 0u, 0u, 0u};
          if (2 * q < cur.cn && k < K && xlive[t]) xb[q][t] = *reinterpret_cast<const u32x4*>(xrow[t] + 32 * (int64_t)(c0 + 2 * q));
        }
    }
    const int c1 = c0 + cur.cn;
    if (c1 < kend) {
      if (c1 - ob + C > kI8OffsetLanes) {
        ob = c1;
        orng = load_offsets(ob);
      }
      ch = shape(orng, c1);
      issue(ch, c1);
    }

    // 3. expand and multiply, one tile pair per MFMA
    const uint32_t vrel = vbuf_addr - cur.a0;
#pragma unroll
    for (int q = 0; q < C / 2; ++q) {
      if (2 * q < cur.cn) {
        const int j = 2 * q + tsel;                            // this lane's tile in the chunk
        uint32_t w = wl[fr * WS + j];
        if (j >= cur.cn) w = 0u;                               // a range ending on half a pair
        // values stored before mine in my tile: a tile's values are ordered by 16-column group (my
        // half), then row (my fr), i.e. in the order of the tile's 32 lanes, so this is the
        // exclusive scan of the kept counts over my half of the wave
        const uint32_t pc = __popc(__builtin_amdgcn_ubfe(w, 16 * half, 16));
        const uint32_t before = half_inclusive_scan(pc) - pc;
        // this lane's tile offset: the pair's first or second (arithmetic select keeps tc[] in registers)
        const uint32_t tile0 = (uint32_t)tc[2 * q] + (((uint32_t)tc[2 * q + 1] - (uint32_t)tc[2 * q]) & (0u - (uint32_t)tsel));
        const uint32_t oa = tile0 + before;
        u32x4 a;
        uint32_t o = oa;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t nib = __builtin_amdgcn_ubfe(w, 16 * half + 4 * i, 4);
          const uint32_t p = o + vrel;
          const uint32_t d = p & ~3u;
          const uint32_t lo = lds_load4(d), hi = lds_load4(d + 4);
          const uint32_t win = __builtin_amdgcn_alignbyte(hi, lo, p);
          const uint32_t sel = lds_load4(lut_addr + 4u * nib);
          a[i] = __builtin_amdgcn_perm(0u, win, sel);
          o += __popc(nib);
        }
        if constexpr (XL) {
          if (xstep) xs_op = lds_load16(xaddr0 + xstep * (uint32_t)((c0 >> 1) + q));
          acc[0] = mfma_i8(a, xs_op, acc[0]);
        } else {
#pragma unroll
          for (int t = 0; t < MT; ++t) acc[t] = mfma_i8(a, xb[q][t], acc[t]);
        }
      }
    }
    wave_lds_sync();
    c0 = c1;
  }
  __syncthreads();
  i8_finish<MT, W>(acc, reinterpret_cast<int32_t*>(dsm), wave, lane, blk * 16, N, m0, M, sx, sw, Y, acc_out);
}

template <int MT>
__global__ void __launch_bounds__(kI8Threads) k_dense_int8(const I8DenseGroupArg g) {
  const int ti = find_task(g.first, g.count);
  const I8DenseTaskArg tk = g.t[ti];
  const int8_t* __restrict__ Xq = tk.Xq;
  const float* __restrict__ sx = tk.sx;
  const int8_t* __restrict__ Wq = tk.W;
  const int64_t M = g.M, K = tk.K, N = tk.N;
  const float* __restrict__ sw = tk.sw;
  uint16_t* __restrict__ Y = tk.Y;
  int32_t* __restrict__ acc_out = tk.acc;
  __shared__ int32_t part[kI8Waves * MT * 256];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int fr = lane & 15, fg = lane >> 4;
  const int Q = (int)((K + 63) / 64);                     // 64-column steps
  const int G = (Q + kI8Unroll - 1) / kI8Unroll;
  const int64_t n0 = ((int64_t)blockIdx.x - g.first[ti]) * 16;
  const int64_t m0 = (int64_t)blockIdx.y * 16 * MT;
  const int64_t wrow = (n0 + fr < N ? n0 + fr : N - 1) * K;
  int64_t xrow[MT];
#pragma unroll
  for (int f = 0; f < MT; ++f) {
    const int64_t m = m0 + 16 * f + fr;
    xrow[f] = (m < M ? m : M - 1) * K;
  }
  i32x4 acc[MT];
#pragma unroll
  for (int f = 0; f < MT; ++f) acc[f] = i32x4{0, 0, 0, 0};
  for (int g = wave; g < G; g += kI8Waves) {
    u32x4 a[kI8Unroll];
    u32x4 xb[kI8Unroll][MT];
#pragma unroll
    for (int u = 0; u < kI8Unroll; ++u) {
      const int q = g * kI8Unroll + u;
      int64_t k = (int64_t)q * 64 + 16 * fg;
      const bool kok = k < K && q < Q;
      if (!kok) k = 0;
      u32x4 v = *reinterpret_cast<const u32x4*>(Wq + wrow + k);
      if (!kok) v = u32x4{0u, 0u, 0u, 0u};
      a[u] = v;
#pragma unroll
      for (int f = 0; f < MT; ++f) {
        u32x4 x = *reinterpret_cast<const u32x4*>(Xq + xrow[f] + k);
        if (!kok) x = u32x4{0u, 0u, 0u, 0u};
        xb[u][f] = x;
      }
    }
#pragma unroll
    for (int u = 0; u < kI8Unroll; ++u)
#pragma unroll
      for (int f = 0; f < MT; ++f) acc[f] = mfma_i8(a[u], xb[u][f], acc[f]);
  }
  i8_finish<MT, kI8Waves>(acc, part, wave, lane, n0, N, m0, M, sx, sw, Y, acc_out);
}

int i8_fragments(int64_t M) { return M <= 16 ? 1 : (M <= 32 ? 2 : 4); }

template <int MT, bool XL, int W>
hipError_t sparse_int8_launch(const I8GroupArg& g, int64_t kmax, hipStream_t s) {
  auto* kernel = k_sparse_int8<MT, XL, W>;
  const size_t region = (size_t)W * kI8VBufAlloc > (size_t)W * MT * 1024 ? (size_t)W * kI8VBufAlloc
                                                                          : (size_t)W * MT * 1024;
  const size_t xbytes = XL ? (size_t)g.M * (size_t)i8_xs_stride(kmax) : 0;
  static PerDeviceFlag lds_set;
  const hipError_t attr = allow_lds_once(lds_set, kernel, region + (XL ? kI8XLdsMax + 16 * 16 : 0));
  if (attr != hipSuccess) return attr;
  const dim3 grid((unsigned)g.first[g.count], (unsigned)((g.M + 16 * MT - 1) / (16 * MT)));
  hipLaunchKernelGGL(kernel, grid, dim3(W * kWave), region + xbytes, s, g);
  return hipGetLastError();
}

// Activations staged in LDS when every task's M x 64 ceil(S/2) bytes fit.
template <int W>
hipError_t sparse_int8_w(const I8GroupArg& g, int64_t kmax, hipStream_t s) {
  const int MT = i8_fragments(g.M);
  if (MT == 1 && (int64_t)g.M * 64 * ((tile_steps(kmax) + 1) / 2) <= kI8XLdsMax)
    return sparse_int8_launch<1, true, W>(g, kmax, s);
  if (MT == 1) return sparse_int8_launch<1, false, W>(g, kmax, s);
  if (MT == 2) return sparse_int8_launch<2, false, W>(g, kmax, s);
  return sparse_int8_launch<4, false, W>(g, kmax, s);
}

// Per-token activation quantisation (paper section 3.4 quantises the
// activations to int8; symmetric, one binary32 scale per row): one workgroup
// per row of X [M][K] (K % 8 == 0, 16-byte pieces of 8 fp16/bf16 values)
// finds amax = max |x| (a wave reduction, then the 4 wave maxima), sets
// scale = amax / 127 (1 when amax is 0), and writes the codes
// clamp(round-half-even(x / scale), -127, 127); each division is correctly
// rounded.  Rows of up to 256 PT pieces stay in registers between the two
// steps (one read of X); PT = 0 re-reads longer rows (from L2).
template <class T, int PT>
__global__ void __launch_bounds__(256) k_quantize_rows(const uint16_t* __restrict__ X, int64_t K,
                                                       int8_t* __restrict__ Xq, float* __restrict__ sx) {
  constexpr int R = PT > 0 ? PT : 1;
  __shared__ float wmax[4];
  const int64_t m = blockIdx.x;
  const uint16_t* x = X + m * K;
  const int64_t P = K / 8;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  auto amax8 = [](const u32x4& v, float a) {
#pragma unroll
    for (int e = 0; e < 8; ++e) a = fmaxf(a, fabsf(T::to_f32((v[e >> 1] >> (16 * (e & 1))) & 0xffffu)));
    return a;
  };
  float amax = 0.0f;
  u32x4 v[R];
  if constexpr (PT > 0) {
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int64_t p = t + 256 * i;
      v[i] = p < P ? *reinterpret_cast<const u32x4*>(x + 8 * p) : u32x4{0u, 0u, 0u, 0u};
      amax = amax8(v[i], amax);
    }
  } else {
    for (int64_t p = t; p < P; p += 256) amax = amax8(*reinterpret_cast<const u32x4*>(x + 8 * p), amax);
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) amax = fmaxf(amax, __shfl_xor(amax, d));
  if (lane == 0) wmax[wave] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
  const float scale = amax == 0.0f ? 1.0f : __fdiv_rn(amax, 127.0f);
  if (t == 0) sx[m] = scale;
  int8_t* q = Xq + m * K;
  auto put8 = [&](const u32x4& w, int64_t p) {
    uint32_t c[2] = {0u, 0u};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float r = rintf(__fdiv_rn(T::to_f32((w[e >> 1] >> (16 * (e & 1))) & 0xffffu), scale));
      r = fminf(fmaxf(r, -127.0f), 127.0f);
      c[e >> 2] |= ((uint32_t)(int32_t)r & 0xffu) << (8 * (e & 3));
    }
    *reinterpret_cast<u32x2*>(q + 8 * p) = u32x2{c[0], c[1]};
  };
  if constexpr (PT > 0) {
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int64_t p = t + 256 * i;
      if (p < P) put8(v[i], p);
    }
  } else {
    for (int64_t p = t; p < P; p += 256) put8(*reinterpret_cast<const u32x4*>(x + 8 * p), p);
  }
}

template <class T>
void quantize_rows_launch(const uint16_t* x, int64_t M, int64_t K, int8_t* Xq, float* sx, hipStream_t s) {
  const int64_t P = K / 8;
  const dim3 grid((unsigned)M), block(256);
  if (P <= 256)
    hipLaunchKernelGGL((k_quantize_rows<T, 1>), grid, block, 0, s, x, K, Xq, sx);
  else if (P <= 512)
    hipLaunchKernelGGL((k_quantize_rows<T, 2>), grid, block, 0, s, x, K, Xq, sx);
  else if (P <= 1024)
    hipLaunchKernelGGL((k_quantize_rows<T, 4>), grid, block, 0, s, x, K, Xq, sx);
  else if (P <= 2048)
    hipLaunchKernelGGL((k_quantize_rows<T, 8>), grid, block, 0, s, x, K, Xq, sx);
  else
    hipLaunchKernelGGL((k_quantize_rows<T, 0>), grid, block, 0, s, x, K, Xq, sx);
}

bool i8_small_grid(int64_t blocks) { return blocks < 2 * (int64_t)device_cus(); }

}  // namespace

hipError_t launch_sparse_int8(const spl_int8_task* tasks, int count, int64_t M, hipStream_t s) {
  if (M >= kI8PrefillMinM) {                         // MFMA-tiled kernel with activations shared in LDS
    for (int i = 0; i < count; ++i) {
      const hipError_t e = launch_sparse_prefill_i8(tasks[i], M, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  I8GroupArg g{};
  g.count = count;
  g.M = (int32_t)M;
  g.first[0] = 0;
  int64_t kmax = 0;
  for (int i = 0; i < count; ++i) {
    const spl_matrix& W = *tasks[i].Wq;
    g.t[i] = I8TaskArg{tasks[i].Xq, tasks[i].x_scales, W.bitmask, static_cast<const uint8_t*>(W.values),
                       W.tile_offsets, W.rows, W.cols, tasks[i].w_scales, static_cast<uint16_t*>(tasks[i].Y),
                       tasks[i].acc_out};
    g.first[i + 1] = g.first[i] + (int32_t)tile_blocks(W.rows);
    kmax = W.cols > kmax ? W.cols : kmax;
  }
  const int64_t blocks = (int64_t)g.first[count] * ((M + 63) / 64);
  return i8_small_grid(blocks) ? sparse_int8_w<16>(g, kmax, s) : sparse_int8_w<8>(g, kmax, s);
}

hipError_t launch_dense_int8(const spl_dense_int8_task* tasks, int count, int64_t M, hipStream_t s) {
  if (M >= kI8PrefillMinM) {
    for (int i = 0; i < count; ++i) {
      const hipError_t e = launch_dense_prefill_i8(tasks[i], M, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  I8DenseGroupArg g{};
  g.count = count;
  g.M = (int32_t)M;
  g.first[0] = 0;
  for (int i = 0; i < count; ++i) {
    g.t[i] = I8DenseTaskArg{tasks[i].Xq, tasks[i].x_scales, tasks[i].Wq, tasks[i].N, tasks[i].K, tasks[i].w_scales,
                            static_cast<uint16_t*>(tasks[i].Y), tasks[i].acc_out};
    g.first[i + 1] = g.first[i] + (int32_t)((tasks[i].N + 15) / 16);
  }
  const int MT = i8_fragments(M);
  const dim3 grid((unsigned)g.first[count], (unsigned)((M + 16 * MT - 1) / (16 * MT))), block(kI8Threads);
  if (MT == 1)
    hipLaunchKernelGGL((k_dense_int8<1>), grid, block, 0, s, g);
  else if (MT == 2)
    hipLaunchKernelGGL((k_dense_int8<2>), grid, block, 0, s, g);
  else
    hipLaunchKernelGGL((k_dense_int8<4>), grid, block, 0, s, g);
  return hipGetLastError();
}

hipError_t launch_quantize_rows_i8(const void* X, int32_t dtype, int64_t M, int64_t K, int8_t* Xq, float* sx,
                                   hipStream_t s) {
  const uint16_t* x = static_cast<const uint16_t*>(X);
  if (dtype == SPL_BF16)
    quantize_rows_launch<Bf16>(x, M, K, Xq, sx, s);
  else
    quantize_rows_launch<F16>(x, M, K, Xq, sx, s);
  return hipGetLastError();
}

}  // namespace spl
