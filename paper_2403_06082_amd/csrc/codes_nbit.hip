// Packing and dequantization of 3- and 4-bit codes (the 2-bit codes have their own kernels
// in the fp64 path).  floor(32 / b) codes per uint32 word, row-major: column j of a row in
// bits b (j mod cpw) .. b (j mod cpw) + b - 1 of word floor(j / cpw), pad bits zero.  The
// paper quantizes at 3 and 4 bits in its appendix on segmentation and detection models;
// the grid and the rounding are those of the 2-bit pass with 2^b levels.
#include "fq_internal.h"

namespace fq {
namespace {

// one thread per output word
__global__ __launch_bounds__(256) void k_pack_nbit(const uint8_t* __restrict__ c8, int64_t rows,
                                                   int64_t cols, int bits,
                                                   uint32_t* __restrict__ out) {
  const int cpw = 32 / bits;
  const uint32_t mask = (1u << bits) - 1u;
  const int64_t nw = (cols + cpw - 1) / cpw;
  const int64_t total = rows * nw;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t r = e / nw, w = e - r * nw;
    const int64_t c0 = w * cpw;
    const uint8_t* src = c8 + r * cols + c0;
    uint32_t word = 0;
    for (int k = 0; k < cpw; ++k)
      if (c0 + k < cols) word |= ((uint32_t)src[k] & mask) << (bits * k);
    out[e] = word;
  }
}

// out[r * ld_out + c] = code[r][c] - zero[r] as bf16 (integers below 2^4 in magnitude,
// exact) for r < rows, c < cols; every other entry of the rows_out x ld_out plane is 0.
// One thread per 16-column group, two 16-byte stores.
__global__ __launch_bounds__(256) void k_dequant_nbit(const uint32_t* __restrict__ codes,
                                                      const float* __restrict__ zero,
                                                      int64_t rows, int64_t cols, int bits,
                                                      u16* __restrict__ out, int64_t ld_out,
                                                      int64_t rows_out) {
  const int cpw = 32 / bits;
  const uint32_t mask = (1u << bits) - 1u;
  const int64_t nw = (cols + cpw - 1) / cpw;     // packed words per code row
  const int64_t gw = ld_out / 16;                // 16-column groups per output row
  const int64_t total = rows_out * gw;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t r = e / gw, g = e - r * gw;
    uint32_t h[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) h[k] = 0;
    if (r < rows) {
      const float z = zero[r];
      const uint32_t* row = codes + r * nw;
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int64_t c = g * 16 + k;
        if (c < cols) {
          const int64_t w = c / cpw;
          const int sh = bits * (int)(c - w * cpw);
          const float v = (float)((row[w] >> sh) & mask) - z;
          h[k] = __float_as_uint(v) >> 16;
        }
      }
    }
    u16* dst = out + r * ld_out + g * 16;
    *reinterpret_cast<uint4*>(dst) = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16),
                                                h[4] | (h[5] << 16), h[6] | (h[7] << 16));
    *reinterpret_cast<uint4*>(dst + 8) = make_uint4(h[8] | (h[9] << 16), h[10] | (h[11] << 16),
                                                    h[12] | (h[13] << 16), h[14] | (h[15] << 16));
  }
}

unsigned grid_of(int64_t n) {
  const int64_t g = (n + 255) / 256;
  return (unsigned)(g < 65536 ? (g > 0 ? g : 1) : 65536);
}

}  // namespace

hipError_t q_pack_nbit(const uint8_t* codes8, int64_t rows, int64_t cols, int bits,
                       uint32_t* out, hipStream_t s) {
  const int cpw = 32 / bits;
  const int64_t nw = rows * ((cols + cpw - 1) / cpw);
  if (nw <= 0) return hipSuccess;
  prof_begin(s, "pack2");
  hipLaunchKernelGGL(k_pack_nbit, dim3(grid_of(nw)), dim3(256), 0, s, codes8, rows, cols, bits, out);
  prof_end(s);
  return last_launch_error();
}

hipError_t dequant_nbit_bf16(const uint32_t* codes, int bits, const float* zero, int64_t rows,
                             int64_t cols, u16* out, int64_t ld_out, int64_t rows_out,
                             hipStream_t s) {
  if (bits == 2) return dequant_bf16(codes, zero, rows, cols, out, ld_out, rows_out, s);
  if (rows_out < rows) rows_out = rows;
  if (ld_out % 16 != 0 || ld_out < cols) return hipErrorInvalidValue;
  const int64_t nw = rows_out * (ld_out / 16);
  if (nw <= 0) return hipSuccess;
  prof_begin(s, "dequant");
  hipLaunchKernelGGL(k_dequant_nbit, dim3(grid_of(nw)), dim3(256), 0, s, codes, zero, rows, cols,
                     bits, out, ld_out, rows_out);
  prof_end(s);
  return last_launch_error();
}

}  // namespace fq
