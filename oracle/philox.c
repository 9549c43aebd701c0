/*
 * Oracle: Philox4x64-10 counter-based generator, written from its published
 * definition (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
 * 1, 2, 3", SC'11, Sec. on the Philox family). TEST INFRASTRUCTURE ONLY.
 *
 * The paper being reproduced draws negatives "from V" at random (Alg. 1) and
 * names subsampling and window parameters (Sec. 2) without fixing a generator;
 * a counter-based generator makes every draw a pure function of
 * (seed, position, epoch, word), so a sequential and a parallel run draw the
 * same numbers.
 */
#include "oracle.h"

/* 64 x 64 -> 128-bit product, written with the compiler's 128-bit integer. */
static void mulhilo64(uint64_t a, uint64_t b, uint64_t* hi, uint64_t* lo) {
  unsigned __int128 p = (unsigned __int128)a * (unsigned __int128)b;
  *hi = (uint64_t)(p >> 64);
  *lo = (uint64_t)p;
}

void oracle_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2],
                          uint64_t out[4]) {
  /* Multipliers and Weyl key increments of Philox4x64 (SC'11, Table 2). */
  const uint64_t M0 = 0xD2E7470EE14C6C93ULL;
  const uint64_t M1 = 0xCA5A826395121157ULL;
  const uint64_t W0 = 0x9E3779B97F4A7C15ULL;
  const uint64_t W1 = 0xBB67AE8584CAA73BULL;
  uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint64_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    uint64_t hi0, lo0, hi1, lo1;
    mulhilo64(M0, x0, &hi0, &lo0);
    mulhilo64(M1, x2, &hi1, &lo1);
    uint64_t y0 = hi1 ^ x1 ^ k0;
    uint64_t y1 = lo1;
    uint64_t y2 = hi0 ^ x3 ^ k1;
    uint64_t y3 = lo0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    k0 += W0;
    k1 += W1;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

uint32_t oracle_draw_u32(uint64_t seed, uint64_t p, uint64_t e, uint32_t word) {
  uint64_t ctr[4] = {p, e, (uint64_t)(word / 8u), 0};
  uint64_t key[2] = {seed, 0};
  uint64_t out[4];
  oracle_philox4x64_10(ctr, key, out);
  uint64_t v = out[(word % 8u) / 2u];
  return (word % 2u) == 0u ? (uint32_t)(v & 0xFFFFFFFFULL) : (uint32_t)(v >> 32);
}
