/* Seeded synthetic contents for the host-resident KV and indexer-key rows.
 *
 * This is an input producer only: it knows nothing about matching, slots or
 * transfers.  Every byte is a pure function of (key, row, byte offset), so any
 * row can be regenerated on demand and both the CPU oracle and the GPU path
 * read identical host memory.
 *
 *   kind 0 (KV row):       bf16 values uniform in [-1, 1), little-endian.
 *   kind 1 (indexer row):  (row_bytes - 4) fp8-e4m3 bytes with finite values,
 *                          followed by one fp32 scale uniform in (0, 1].
 *
 * The mixing function is splitmix64 (Steele, Lea, Flood; "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), applied to a counter.
 */
#include <stdint.h>
#include <string.h>

static inline uint64_t splitmix64(uint64_t z) {
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static inline uint16_t bf16_from_u16(uint16_t u) {
    /* u / 65536 * 2 - 1 lies in [-1, 1) and is exact in fp32; truncating to
     * bf16 rounds toward zero, which keeps the value inside [-1, 1). */
    float f = (float)u * (1.0f / 32768.0f) - 1.0f;
    uint32_t b;
    memcpy(&b, &f, 4);
    return (uint16_t)(b >> 16);
}

static inline uint8_t fp8_e4m3_finite(uint8_t v) {
    /* e4m3 encodes NaN as S.1111.111; map those two codes to the largest
     * finite magnitude so every byte is a valid finite value. */
    return ((v & 0x7Fu) == 0x7Fu) ? (uint8_t)(v & 0xFEu) : v;
}

static void fill_row(uint8_t *dst, int64_t row, int64_t row_bytes, int kind, uint64_t key) {
    uint64_t base = splitmix64(key ^ splitmix64((uint64_t)row));
    if (kind == 0) {
        int64_t nwords = row_bytes / 8;
        for (int64_t w = 0; w < nwords; ++w) {
            uint64_t r = splitmix64(base + (uint64_t)w);
            uint16_t h[4];
            for (int k = 0; k < 4; ++k) h[k] = bf16_from_u16((uint16_t)(r >> (16 * k)));
            memcpy(dst + 8 * w, h, 8);
        }
        for (int64_t b = nwords * 8; b < row_bytes; b += 2) {
            uint64_t r = splitmix64(base + 0x100000000ull + (uint64_t)b);
            uint16_t h = bf16_from_u16((uint16_t)r);
            memcpy(dst + b, &h, (row_bytes - b) >= 2 ? 2 : 1);
        }
    } else {
        int64_t payload = row_bytes - 4;
        for (int64_t b = 0; b < payload; b += 8) {
            uint64_t r = splitmix64(base + (uint64_t)b);
            for (int k = 0; k < 8 && b + k < payload; ++k)
                dst[b + k] = fp8_e4m3_finite((uint8_t)(r >> (8 * k)));
        }
        uint64_t r = splitmix64(base + 0x200000000ull);
        float scale = (float)((r >> 40) + 1) * (1.0f / 16777216.0f); /* (0, 1] */
        memcpy(dst + payload, &scale, 4);
    }
}

/* Fill rows [first_row, first_row + n_rows) of a row-major region whose row 0
 * starts at base.  Returns 0, or -1 on bad arguments. */
int avsg_wl_fill_rows(void *base, int64_t first_row, int64_t n_rows, int64_t row_bytes,
                      int kind, uint64_t key, int nthreads) {
    if (!base || n_rows < 0 || first_row < 0 || row_bytes <= 0) return -1;
    if (kind != 0 && kind != 1) return -1;
    if (kind == 1 && row_bytes < 8) return -1;
    uint8_t *p = (uint8_t *)base;
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1)
    for (int64_t i = 0; i < n_rows; ++i) {
        int64_t row = first_row + i;
        fill_row(p + row * row_bytes, row, row_bytes, kind, key);
    }
    return 0;
}

/* Key derivation shared by every caller: (seed, config id, stream, request,
 * version) -> 64-bit key.  Version 0 is the initial fill; a positive version
 * is a regeneration of speculative positions. */
uint64_t avsg_wl_key(uint64_t seed, uint64_t cfg_id, uint64_t stream, uint64_t request,
                     uint64_t version) {
    uint64_t k = splitmix64(seed);
    k = splitmix64(k ^ (cfg_id * 0x100000001B3ull));
    k = splitmix64(k ^ (stream + 0x51ull));
    k = splitmix64(k ^ (request * 0x9E3779B1ull));
    k = splitmix64(k ^ (version * 0xC2B2AE3D27D4EB4Full));
    return k;
}
