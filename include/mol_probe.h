/*
 * mol_probe.h -- measurement aid of the MoL library (not part of the
 * retrieval ABI in mol.h): the issue-rate floor of the fused scan's
 * instruction mix on gfx950.
 *
 * One "wave-step" of the fused exact scan (k_mol_fused, Px = 8, d = 64,
 * H = 64: 2 queries x 16 items per wave) issues 48 matrix instructions
 * (v_mfma_f32_16x16x32 bf16/f16), 97 transcendental vector instructions
 * (the SiLU's exp2 and reciprocal, the softmax's exp2, the reciprocal of
 * phi) and 238 other vector ALU instructions, 32 of them f32 -> f16 pack
 * conversions (the counts of the SQ_INSTS_* hardware counters per
 * wave-step).  The probe
 * kernel issues exactly that mix per iteration with no data dependencies
 * between the instructions, no memory traffic and no synchronisation, so its
 * time per wave-step is a floor for any schedule of the same instructions.
 *
 *   pattern 0: the mix, each MFMA followed by its share of vector work
 *   pattern 1: the vector ALU part alone (no MFMA)
 *   pattern 2: the MFMA part alone
 *   pattern 3: the mix in two phases per iteration (48 MFMAs, then the rest)
 *   pattern 4: pattern 0 plus the rest of the kernel's per-step stream: 28
 *              LDS reads of 16 bytes per lane, 39 scalar ALU instructions and
 *              the listing's hazard nops: two 11-slot MFMA drains and 25
 *              three-slot nops (still no dependencies)
 *
 * The launch holds waves_per_simd waves on each of the 1024 SIMDs
 * (256 x waves_per_simd workgroups of 4 waves); each wave runs `iters`
 * wave-steps.  sink: DEVICE buffer of 256 * waves_per_simd * 256 floats
 * (written, to keep the instructions live).  Asynchronous on `stream`
 * (hipStream_t as void*); returns 0, or a nonzero HIP error code for a
 * launch failure; waves_per_simd outside 1..8, iters < 1 or an unknown
 * pattern return -1 with nothing launched.
 */
#ifndef MOL_PROBE_H
#define MOL_PROBE_H
#ifdef __cplusplus
extern "C" {
#endif

int mol_probe_issue_mix(int pattern, int waves_per_simd, int iters, float *sink, void *stream);

#ifdef __cplusplus
}
#endif
#endif
