/*
 * Seeded synthetic inputs: the counter-based generator behind every test and
 * benchmark input (weights, KV-pool contents, the fragmented live map and the
 * corruption site).  It holds none of the restore/verify arithmetic.
 *
 * Philox4x32-10 follows its published definition: Salmon, Moraes, Dror and
 * Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3", SC'11 (multipliers
 * 0xD2511F53 / 0xCD9E8D57, Weyl key bumps 0x9E3779B9 / 0xBB67AE85, ten
 * rounds).  Its known-answer vectors are the Random123 ones.
 *
 * The same source is compiled for the host (gcc, synth_host.c) and for the
 * GPU (hipcc, synth_dev.hip), so both sides draw bit-identical values.  The
 * includer defines SYNTH_FN with the qualifiers its compiler needs.
 *
 * Weight values are bf16 drawn as an approximate N(0, 0.02): the sum of four
 * uniform 16-bit integers (Irwin-Hall, n = 4) centred at zero, scaled by one
 * IEEE f32 multiply, then rounded to bf16 (nearest-even) with integer
 * operations.  Everything except the multiply is integer arithmetic and the
 * multiply's operand is an exactly representable integer, so the host and
 * the GPU produce the same bits.
 */
#ifndef SYNTH_PHILOX_H
#define SYNTH_PHILOX_H

#include <stdint.h>

#ifndef SYNTH_FN
#error "define SYNTH_FN (function qualifiers) before including philox.h"
#endif

#define SYNTH_PHILOX_M0 0xD2511F53u
#define SYNTH_PHILOX_M1 0xCD9E8D57u
#define SYNTH_PHILOX_W0 0x9E3779B9u
#define SYNTH_PHILOX_W1 0xBB67AE85u

/* 0.02 / std(sum of four U{0..65535}) rounded to f32: bits 0x350DE3BD. */
#define SYNTH_BF16_SCALE_BITS 0x350DE3BDu
/* Mean of the sum of four U{0..65535}. */
#define SYNTH_IH4_MEAN 131070

typedef struct { uint32_t v[4]; } synth_u32x4;

SYNTH_FN synth_u32x4 synth_philox4x32_10(synth_u32x4 ctr, uint32_t k0, uint32_t k1)
{
    for (int r = 0; r < 10; ++r) {
        uint64_t p0 = (uint64_t)SYNTH_PHILOX_M0 * ctr.v[0];
        uint64_t p1 = (uint64_t)SYNTH_PHILOX_M1 * ctr.v[2];
        synth_u32x4 n;
        n.v[0] = (uint32_t)(p1 >> 32) ^ ctr.v[1] ^ k0;
        n.v[1] = (uint32_t)p1;
        n.v[2] = (uint32_t)(p0 >> 32) ^ ctr.v[3] ^ k1;
        n.v[3] = (uint32_t)p0;
        ctr = n;
        k0 += SYNTH_PHILOX_W0;
        k1 += SYNTH_PHILOX_W1;
    }
    return ctr;
}

/* One 128-bit draw addressed by (stream, index) under a 64-bit seed. */
SYNTH_FN synth_u32x4 synth_draw(uint64_t seed, uint64_t stream, uint64_t index)
{
    synth_u32x4 c;
    c.v[0] = (uint32_t)index;
    c.v[1] = (uint32_t)(index >> 32);
    c.v[2] = (uint32_t)stream;
    c.v[3] = (uint32_t)(stream >> 32);
    return synth_philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
}

/* Four 16-bit uniforms from two 32-bit draws -> bf16 bits of ~N(0, 0.02). */
SYNTH_FN uint16_t synth_bf16_from_u32x2(uint32_t a, uint32_t b)
{
    int32_t s = (int32_t)((a & 0xFFFFu) + (a >> 16) + (b & 0xFFFFu) + (b >> 16)) - SYNTH_IH4_MEAN;
    union { uint32_t u; float f; } scale, val;
    scale.u = SYNTH_BF16_SCALE_BITS;
    val.f = (float)s * scale.f;
    uint32_t u = val.u;
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/* Element e of tensor t under seed: one Philox draw serves elements 2k, 2k+1. */
SYNTH_FN uint16_t synth_bf16(uint64_t seed, uint64_t tensor, uint64_t elem)
{
    synth_u32x4 r = synth_draw(seed, tensor, elem >> 1);
    return (elem & 1) ? synth_bf16_from_u32x2(r.v[2], r.v[3])
                      : synth_bf16_from_u32x2(r.v[0], r.v[1]);
}

#endif
