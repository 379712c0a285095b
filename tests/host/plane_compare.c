/* Byte-for-byte comparison of one slab of stored planes with the bytes the
 * oracle's residues and limb tables give, for the full-size GPU parity
 * tests (tests/plane_check.py).  Test infrastructure: table lookups and
 * equality only, no step of the method.
 *
 *  R:      int16 [r][nv][k]     the oracle's centred residues of the slab
 *  tab:    uint8 [sum_i m_i][3] per modulus i, at rows tab_off[i] + d + m_i/2,
 *                               the stored bytes of residue d (limbs 0..nl_i-1)
 *  got:    uint8 [np][nv][kp]   the library's planes of the slab, kp >= k;
 *                               plane q0_i + p holds limb p of modulus i
 *  Returns the number of differing bytes (the padding l >= k must be zero)
 *  and the flat index into got of the first one in *first (-1 if none). */
#include <stdint.h>

int64_t plane_compare(int r, const int64_t* mods, const int* nlimbs, const int64_t* tab_off,
                      const uint8_t* tab, int64_t nv, int64_t k, int64_t kp, const int16_t* R,
                      const uint8_t* got, int64_t* first) {
  int64_t bad = 0;
  *first = -1;
  int q0 = 0;
  for (int i = 0; i < r; ++i) {
    const int64_t half = mods[i] / 2;
    for (int p = 0; p < nlimbs[i]; ++p) {
      const uint8_t* g = got + (int64_t)(q0 + p) * nv * kp;
      for (int64_t v = 0; v < nv; ++v) {
        const int16_t* rv = R + ((int64_t)i * nv + v) * k;
        const uint8_t* gv = g + v * kp;
        for (int64_t l = 0; l < kp; ++l) {
          const uint8_t want = l < k ? tab[(tab_off[i] + rv[l] + half) * 3 + p] : 0;
          if (gv[l] != want) {
            if (*first < 0) *first = (gv - got) + l;
            ++bad;
          }
        }
      }
    }
    q0 += nlimbs[i];
  }
  return bad;
}
