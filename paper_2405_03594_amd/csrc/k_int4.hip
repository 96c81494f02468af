// 4-bit sparse payloads (paper section 4 lists INT4 among the next steps) for
// the sparse-quantized linear layer at decode batches (M <= 16).
//
// Storage: the pattern of the int8 tile layout (bitmask words, tile offsets;
// values ordered by 16-column group, then row, then column) with value i held
// as the two's-complement nibble at byte i / 2, low nibble first.  The codes
// are the int8 path's integers restricted to [-8, 7], so the products (exact
// int32 sums on v_mfma_i32_16x16x64_i8) and the epilogue are those of the
// int8 path:  Y[m][n] = fp16_rne((float(acc) * sx[m]) * sw[n]).
//
// Kernel: one workgroup per 16-row block, its W waves (8, or 16 when the
// launch has fewer than two row blocks per CU) over contiguous ranges
// of tile pairs (one MFMA each: lanes 0-31 tile 2p, lanes 32-63 tile 2p + 1,
// lane (fr, fg) row fr, columns 16 (fg % 2) .. + 16 of its tile).  A lane's
// first value is nibble toff[t] + the exclusive scan of its tile half's kept
// counts; its (at most 16) nibbles are read as three aligned dwords, shifted
// into place with v_alignbit_b32; for each 4-column nibble of its mask the 4
// nibbles from the nibble's first rank are widened to sign-extended bytes and
// a 16-entry selector table (v_perm_b32) places them, zeros where the bitmask
// is clear.  Activation rows
// are read directly (16 bytes per lane), int32 partial sums added in LDS.
// Each wave pipelines its pairs so that no global load is waited for in the
// pair that issues it: pattern words and tile offsets two pairs ahead, nibble
// dwords and activations one pair ahead.
#include "spl_common.h"

namespace spl {
namespace {


// Four nibbles (bits 0-15) -> four sign-extended bytes.
__device__ __forceinline__ uint32_t i4_widen(uint32_t w) {
  uint32_t y = (w & 0xFu) | ((w & 0xF0u) << 4) | ((w & 0xF00u) << 8) | ((w & 0xF000u) << 12);
  const uint32_t m = y & 0x08080808u;                // sign bits
  return y | ((m << 5) - (m << 1));                  // 0xF0 into every byte whose sign bit is set (mod 2^32)
}

__device__ __forceinline__ i32x4 mfma_i8_i4(u32x4 a, u32x4 b, i32x4 c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, a), __builtin_bit_cast(i32x4, b), c, 0, 0,
                                               0);
}

__global__ void __launch_bounds__(256) k_pack_nibbles(const int8_t* __restrict__ v8, int64_t nnz,
                                                      uint8_t* __restrict__ v4, int32_t* __restrict__ bad) {
  const int64_t nb = (nnz + 1) / 2;
  int32_t outside = 0;   // codes of this thread outside [-8, 7]
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nb; i += (int64_t)gridDim.x * 256) {
    const int32_t a = v8[2 * i];
    const int32_t b = 2 * i + 1 < nnz ? (int32_t)v8[2 * i + 1] : 0;
    outside += (a < -8 || a > 7) + (b < -8 || b > 7);
    v4[i] = (uint8_t)(((uint32_t)a & 0xFu) | (((uint32_t)b & 0xFu) << 4));
  }
  if (bad && outside) atomicAdd(bad, outside);
}

__global__ void k_clear_count(int32_t* c) { *c = 0; }

struct I4Args {
  const int8_t* Xq;          // [M][K]
  const float* sx;           // [M]
  const uint32_t* bm;        // [B*S][16]
  const uint8_t* v4;         // nibbles (followed by 16 readable bytes)
  const int32_t* toff;       // [B*S + 1]
  const float* sw;           // [N]
  uint16_t* Y;               // [M][N] fp16
  int32_t* acc_out;          // optional [M][N]
  int64_t N, K;
  int32_t M;
};

template <int W>
__global__ void __launch_bounds__(W * 64) k_sparse_i4(const I4Args g) {
  __shared__ i32x4 part[W][64];
  __shared__ uint32_t sel4[16];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, fr = lane & 15, fg = lane >> 4;
  if (threadIdx.x < 16) sel4[threadIdx.x] = nibble_selector8(threadIdx.x);
  __syncthreads();
  const int64_t b = blockIdx.x;
  const int S = (int)tile_steps(g.K);
  const int P = (S + 1) / 2;                         // tile pairs (64 columns each)
  const int L = (P + W - 1) / W;
  const int pb = wave * L < P ? wave * L : P;
  const int pe = pb + L < P ? pb + L : P;
  const bool xlive = fr < g.M;
  // Software pipeline over tile pairs: the pattern word and tile offset of
  // pair p + 2, the nibble dwords and activation row of pair p + 1 are in
  // flight while pair p is expanded and multiplied (the nibble addresses need
  // the scan of that pair's counts, so they are issued one pair behind the
  // pattern loads).
  // Every load is issued unconditionally (raw buffer loads: an offset past a
  // buffer's size returns zeros), so each pair issues the same loads and the
  // waits before its MFMA cover only the loads of earlier pairs.
  struct Meta {
    uint32_t w, base;   // my tile row's bitmask word (both halves), the tile's first value
  };
  struct Vals {
    uint32_t hw, d0, d1, d2, sh;
  };
  const int h = fg & 1;
  // this row block's words and tile offsets; tiles past S (odd S) and pairs past the range read zeros
  const __amdgpu_buffer_rsrc_t bm_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(g.bm + b * S * 16), (short)0, 64 * S, 0x00020000);
  const __amdgpu_buffer_rsrc_t to_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int32_t*>(g.toff + b * S), (short)0, 4 * S, 0x00020000);
  const __amdgpu_buffer_rsrc_t x_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int8_t*>(g.Xq), (short)0, (int)(g.M * g.K), 0x00020000);
  constexpr uint32_t kOob = 0x80000000u;             // past every buffer above (the host bounds them)
  auto load_meta = [&](int p) {
    const uint32_t s = (uint32_t)(2 * p + (fg >> 1));
    const bool ok = p < pe;
    Meta m;
    m.w = __builtin_amdgcn_raw_buffer_load_b32(bm_rsrc, ok ? 4u * (16u * s + (uint32_t)fr) : kOob, 0, 0);
    m.base = __builtin_amdgcn_raw_buffer_load_b32(to_rsrc, ok ? 4u * s : kOob, 0, 0);
    return m;
  };
  // needs every lane (the half-wave scan); the loads are unconditional: a lane
  // with no kept value reads the dwords at its offset, which lie inside the
  // values buffer (off <= nnz, and nnz / 2 + 16 bytes are readable)
  auto load_vals = [&](const Meta& m) {
    Vals v;
    v.hw = (m.w >> (16 * h)) & 0xffffu;
    const uint32_t cnt = __popc(v.hw);
    const uint32_t off = m.base + half_inclusive_scan(cnt) - cnt;   // nibble index of my first value
    const uint32_t byte0 = off >> 1;
    const uint32_t* d = reinterpret_cast<const uint32_t*>(g.v4 + (byte0 & ~3u));
    v.d0 = d[0];
    v.d1 = d[1];
    v.d2 = d[2];
    v.sh = (byte0 & 3u) * 8u + (off & 1u) * 4u;       // 0 .. 28
    return v;
  };
  auto load_x = [&](int p) {
    const uint32_t k0 = 64u * (uint32_t)p + 16u * (uint32_t)fg;
    const bool ok = p < pe && xlive && (int64_t)k0 < g.K;                             // K % 16 == 0
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                         x_rsrc, ok ? (uint32_t)fr * (uint32_t)g.K + k0 : kOob, 0, 0));
  };
  auto mul = [&](const Vals& v, const u32x4& x, i32x4& acc) {
    u32x4 a = u32x4{0u, 0u, 0u, 0u};
    if (v.hw != 0u) {
      const uint32_t lo = __builtin_amdgcn_alignbit(v.d1, v.d0, v.sh);   // nibbles off .. off + 7
      const uint32_t hi = __builtin_amdgcn_alignbit(v.d2, v.d1, v.sh);   // nibbles off + 8 .. off + 15
      const uint64_t nibs = ((uint64_t)hi << 32) | lo;
      uint32_t rank = 0u;                            // values before this 4-column nibble
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t m4 = (v.hw >> (4 * q)) & 0xFu;
        const uint32_t y = i4_widen((uint32_t)(nibs >> (4u * rank)) & 0xFFFFu);   // ranks rank .. rank + 3
        a[q] = __builtin_amdgcn_perm(0u, y, sel4[m4]);
        rank += __popc(m4);
      }
    }
    acc = mfma_i8_i4(a, x, acc);
  };
  // two pairs per iteration with the roles of the register sets swapped, so
  // that no loaded register is copied (a copy would wait for its load); a pair
  // past the range has zero words and activations and adds nothing
  i32x4 acc = i32x4{0, 0, 0, 0};
  Meta m1 = load_meta(pb + 1);
  Vals v0 = load_vals(load_meta(pb));
  u32x4 x0 = load_x(pb);
  for (int p = pb; p < pe; p += 2) {
    const Meta m2 = load_meta(p + 2);
    const Vals v1 = load_vals(m1);
    const u32x4 x1 = load_x(p + 1);
    mul(v0, x0, acc);
    m1 = load_meta(p + 3);
    v0 = load_vals(m2);
    x0 = load_x(p + 2);
    mul(v1, x1, acc);
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave != 0) return;
  i32x4 sum = part[0][lane];
#pragma unroll
  for (int w = 1; w < W; ++w) sum += part[w][lane];
  const int m = lane & 15;
  if (m >= g.M) return;
  const float xs = g.sx[m];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t n = b * 16 + 4 * (lane >> 4) + r;
    if (n >= g.N) continue;
    const int32_t v = sum[r];
    if (g.acc_out) g.acc_out[(int64_t)m * g.N + n] = v;
    g.Y[(int64_t)m * g.N + n] = F16::from_f32(__fmul_rn(__fmul_rn((float)v, xs), g.sw[n]));
  }
}

}  // namespace

int64_t int4_values_bytes(int64_t nnz) { return spl_values_bytes(SPL_I4, nnz); }

hipError_t launch_pack_nibbles(const int8_t* v8, int64_t nnz, uint8_t* v4, int32_t* bad, hipStream_t s) {
  int64_t blocks = ((nnz + 1) / 2 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  if (bad) hipLaunchKernelGGL(k_clear_count, dim3(1), dim3(1), 0, s, bad);
  hipLaunchKernelGGL(k_pack_nibbles, dim3((unsigned)blocks), dim3(256), 0, s, v8, nnz, v4, bad);
  return hipGetLastError();
}

hipError_t launch_sparse_int4(const int8_t* Xq, const float* sx, int64_t M, const spl_matrix& W4, const float* sw,
                              void* Y, int32_t* acc_out, hipStream_t s) {
  // the kernel addresses X, a row block's words and its tile offsets with 32-bit buffer offsets
  if (M * W4.cols >= (int64_t)1 << 31 || tile_steps(W4.cols) >= (int64_t)1 << 25) return hipErrorNotSupported;
  I4Args g{Xq, sx, W4.bitmask, static_cast<const uint8_t*>(W4.values), W4.tile_offsets, sw,
           static_cast<uint16_t*>(Y), acc_out, W4.rows, W4.cols, (int32_t)M};
  const int64_t blocks = tile_blocks(W4.rows);
  if (blocks < 2 * (int64_t)device_cus())
    hipLaunchKernelGGL(k_sparse_i4<16>, dim3((unsigned)blocks), dim3(16 * 64), 0, s, g);
  else
    hipLaunchKernelGGL(k_sparse_i4<8>, dim3((unsigned)blocks), dim3(8 * 64), 0, s, g);
  return hipGetLastError();
}

}  // namespace spl
