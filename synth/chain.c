/* Chained block hashes for the synthetic trace generator (generator side only).
 *
 * Content id of block j of a segment with key k: c_j = mix64(k ^ (j + 1) * G);
 * chained hash: h_j = mix64(h_{j-1} ^ c_j), with 0 and 2^64-1 (reserved by the
 * block index) remapped to 1.  mix64 is the SplitMix64 finalizer (Steele, Lea
 * and Flood, 2014).
 */
#include <stdint.h>

static uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Hashes of n blocks of one segment chained from parent hash h; returns the
 * last hash (h itself when n = 0). */
uint64_t synth_chain_segment(uint64_t h, uint64_t key, int64_t n, uint64_t *out)
{
    const uint64_t G = 0x9E3779B97F4A7C15ull;
    for (int64_t j = 0; j < n; ++j) {
        uint64_t c = mix64(key ^ ((uint64_t)(j + 1) * G));
        h = mix64(h ^ c);
        if (h == 0 || h == ~0ull) h = 1;
        out[j] = h;
    }
    return h;
}
