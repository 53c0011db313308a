/*
 * synth.hip -- fills rank arenas with the seeded states of synth.h, on the
 * GPU (large workloads) or on the host (small ones and CPU tests).
 * Test and benchmark infrastructure; see synth.h.
 */
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include "synth.h"

static uint64_t seed_mix_of(uint32_t seed) { return synth_mix64((uint64_t)seed); }

/* element l of the piece (row-major in the local box) -> 4 kinds */
__global__ void synth_fill_piece_kernel(synth_piece p, uint64_t seed_mix, uint16_t* a0,
                                        uint32_t* a1, uint32_t* a2, uint32_t* a3) {
  const int64_t ld = p.c1 - p.c0;
  const uint64_t n = (uint64_t)((p.r1 - p.r0) * ld);
  for (uint64_t l = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; l < n;
       l += (uint64_t)gridDim.x * blockDim.x) {
    const int64_t r = p.r0 + (int64_t)(l / (uint64_t)ld);
    const int64_t c = p.c0 + (int64_t)(l % (uint64_t)ld);
    const uint64_t idx = (uint64_t)(r * p.full_cols + c);
    const uint32_t master = synth_f32_bits(seed_mix, 1, p.tensor, idx);
    a0[p.off + l] = synth_bf16_rne(master);
    a1[p.off + l] = master;
    a2[p.off + l] = synth_f32_bits(seed_mix, 2, p.tensor, idx);
    a3[p.off + l] = synth_f32_bits(seed_mix, 3, p.tensor, idx);
  }
}

extern "C" {

/* Fill the payload of n pieces into device arenas (4 kinds) on `stream`.
 * Returns 0, or a hipError_t value. */
int synth_fill_device(const synth_piece* pieces, int n, void* const arenas[4], uint32_t seed,
                      void* stream) {
  const uint64_t sm = seed_mix_of(seed);
  for (int i = 0; i < n; ++i) {
    const synth_piece p = pieces[i];
    const uint64_t ne = (uint64_t)((p.r1 - p.r0) * (p.c1 - p.c0));
    if (ne == 0) continue;
    uint64_t blocks = (ne + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(synth_fill_piece_kernel, dim3((unsigned)blocks), dim3(256), 0,
                       (hipStream_t)stream, p, sm, (uint16_t*)arenas[0], (uint32_t*)arenas[1],
                       (uint32_t*)arenas[2], (uint32_t*)arenas[3]);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
  }
  return 0;
}

/* Same fill into host arenas. */
int synth_fill_host(const synth_piece* pieces, int n, void* const arenas[4], uint32_t seed) {
  const uint64_t sm = seed_mix_of(seed);
  uint16_t* a0 = (uint16_t*)arenas[0];
  uint32_t* a1 = (uint32_t*)arenas[1];
  uint32_t* a2 = (uint32_t*)arenas[2];
  uint32_t* a3 = (uint32_t*)arenas[3];
  for (int i = 0; i < n; ++i) {
    const synth_piece p = pieces[i];
    const int64_t ld = p.c1 - p.c0;
    const uint64_t ne = (uint64_t)((p.r1 - p.r0) * ld);
    for (uint64_t l = 0; l < ne; ++l) {
      const int64_t r = p.r0 + (int64_t)(l / (uint64_t)ld);
      const int64_t c = p.c0 + (int64_t)(l % (uint64_t)ld);
      const uint64_t idx = (uint64_t)(r * p.full_cols + c);
      const uint32_t master = synth_f32_bits(sm, 1, p.tensor, idx);
      a0[p.off + l] = synth_bf16_rne(master);
      a1[p.off + l] = master;
      a2[p.off + l] = synth_f32_bits(sm, 2, p.tensor, idx);
      a3[p.off + l] = synth_f32_bits(sm, 3, p.tensor, idx);
    }
  }
  return 0;
}

/* Values of one kind at logical indices idx[0..n) of a tensor (host).
 * out holds uint16 (kind 0) or uint32 (kinds 1..3). */
int synth_values(uint32_t seed, int kind, int tensor, const uint64_t* idx, int64_t n, void* out) {
  const uint64_t sm = seed_mix_of(seed);
  for (int64_t j = 0; j < n; ++j) {
    if (kind == 0)
      ((uint16_t*)out)[j] = synth_bf16_rne(synth_f32_bits(sm, 1, tensor, idx[j]));
    else
      ((uint32_t*)out)[j] = synth_f32_bits(sm, kind, tensor, idx[j]);
  }
  return 0;
}

}  // extern "C"
