// One-time permutation of row-major bf16 expert weights into the packed
// layout of BASE_W_PACKED (see base_pack_experts in base.h): fragments of
// 16 rows x 32 contraction elements stored lane by lane (64 x 8 elements),
// rows grouped four 16-row tiles at a time, order
// [E][group][k-step][tile][fragment].
#include "common.hpp"
#include "internal.hpp"

namespace basek {

// One thread moves one 16-byte lane slice.  Destination order
// [E][group][k-step][tile 0..3][lane 0..63][8 elements]; source row of
// (group g, tile t): w13 (gate_up = 1): (t < 2 ? 0 : I) + 32 g + 16 (t & 1);
// w2 (gate_up = 0): 64 g + 16 t; plus lane % 16.
__global__ __launch_bounds__(256)
void k_pack(const uint16_t *__restrict__ src, uint16_t *__restrict__ dst,
            long long total_slices, int rows_per_e, int kdim, int groups,
            int I, int gate_up) {
  const long long q = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= total_slices) return;
  const int lane = (int)(q % 64);
  const int t = (int)((q / 64) % 4);
  const int ksteps = kdim / 32;
  const int ks = (int)((q / 256) % ksteps);
  const long long gq = q / (256LL * ksteps);
  const int g = (int)(gq % groups);
  const long long u = gq / groups;
  const int row0 = gate_up ? (t < 2 ? 0 : I) + 32 * g + 16 * (t & 1) : 64 * g + 16 * t;
  const int row = row0 + (lane & 15);
  const int k = 32 * ks + 8 * (lane >> 4);
  const u32x4 v = *reinterpret_cast<const u32x4 *>(
      src + ((size_t)u * rows_per_e + row) * kdim + k);
  *reinterpret_cast<u32x4 *>(dst + (size_t)q * 8) = v;
}

hipError_t launch_pack(const void *w13, const void *w2, void *w13p, void *w2p,
                       int E, int d, int I, hipStream_t st) {
  const long long s13 = (long long)E * 2 * I * d / 8;
  launch_k(k_pack, dim3((unsigned)((s13 + 255) / 256)), dim3(256), 0,
                     st, (const uint16_t *)w13, (uint16_t *)w13p, s13, 2 * I, d,
                     I / 32, I, 1);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long long s2 = (long long)E * d * I / 8;
  launch_k(k_pack, dim3((unsigned)((s2 + 255) / 256)), dim3(256), 0,
                     st, (const uint16_t *)w2, (uint16_t *)w2p, s2, d, I, d / 64, I, 0);
  return hipGetLastError();
}

}  // namespace basek
