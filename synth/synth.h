/*
 * synth.h -- seeded synthetic optimizer/model states, the input generator
 * shared by the tests and the benchmark.
 *
 * Test and benchmark infrastructure: it holds none of the resharding
 * arithmetic.  Its one job is to say what value a logical state element has,
 * so that every replica of an element, on every rank and in every
 * configuration, carries identical bits (as real training states do).
 *
 * value(seed, kind, tensor, idx), idx = row * full_cols + col of the element
 * in its full (TP = 1) tensor:
 *   h  = SplitMix64(SplitMix64(seed) ^ ctr)      ctr = kind<<60 | tensor<<36 | idx
 *        (SplitMix64 finalizer: Steele, Lea and Flood, OOPSLA 2014)
 *   S  = sum of the four 16-bit fields of h, minus 2*65535  (Irwin-Hall, n = 4)
 *   z  = (double)S * C_sigma, rounded once to fp32 (RNE)
 *        C_sigma = sigma / sqrt(4 * (65536^2 - 1) / 12), so z has std sigma
 * kinds: 1 fp32 master ~ N(0, 0.02); 2 fp32 Adam m ~ N(0, 0.02);
 *        3 fp32 Adam v = |N(0, 1e-4)|; 0 bf16 param = RNE-to-bf16 of kind 1.
 * Only integer operations, one exact int->double conversion, one correctly
 * rounded double multiply and one double->float rounding are used, so the
 * host and the GPU produce identical bits.
 */
#ifndef SYNTH_H
#define SYNTH_H
#include <stdint.h>

#ifdef __HIPCC__
#define SYNTH_FN __host__ __device__ static inline
#else
#define SYNTH_FN static inline
#endif

#define SYNTH_C_SIGMA_002 0x1.1bc779ef9b324p-21  /* 0.02 / 37837.227... */
#define SYNTH_C_SIGMA_1EM4 0x1.6b3cc509bc694p-29 /* 1e-4 / 37837.227... */

/* placement of one local piece of a logical tensor inside a rank's arenas */
typedef struct {
  int32_t tensor;
  int32_t reserved;
  int64_t full_cols;      /* columns of the full logical tensor            */
  int64_t r0, r1, c0, c1; /* box in full-tensor coordinates                */
  uint64_t off;           /* element offset of the piece in all 4 arenas   */
} synth_piece;

SYNTH_FN uint64_t synth_mix64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* fp32 bits of kind 1..3 at logical index idx of tensor `tensor` */
SYNTH_FN uint32_t synth_f32_bits(uint64_t seed_mix, int kind, int tensor, uint64_t idx) {
  const uint64_t ctr = ((uint64_t)kind << 60) | ((uint64_t)tensor << 36) | idx;
  const uint64_t h = synth_mix64(seed_mix ^ ctr);
  const int32_t s = (int32_t)(h & 0xFFFF) + (int32_t)((h >> 16) & 0xFFFF) +
                    (int32_t)((h >> 32) & 0xFFFF) + (int32_t)(h >> 48) - 2 * 65535;
  const double c = kind == 3 ? SYNTH_C_SIGMA_1EM4 : SYNTH_C_SIGMA_002;
  const float z = (float)((double)s * c);
  union {
    float f;
    uint32_t u;
  } v;
  v.f = z;
  if (kind == 3) v.u &= 0x7FFFFFFFu;
  return v.u;
}

/* round-to-nearest-even fp32 -> bf16 on the bits (inputs are finite) */
SYNTH_FN uint16_t synth_bf16_rne(uint32_t f) {
  return (uint16_t)((f + 0x7FFFu + ((f >> 16) & 1u)) >> 16);
}

#endif
