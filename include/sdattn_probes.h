/*
 * sdattn_probes.h -- C ABI of libsdattn_probes.so, the measurement kernels
 * behind the denominators the benchmark reports beside the datasheet peaks
 * (sustained fp16 matrix-core rate and shader clock on near-constant and on
 * random operands, the exponential and FMA rates and how each shares a SIMD
 * with the matrix core, the self-attention tile's instruction mix, HBM
 * streaming rates, and a plain copy with the cross-attention kernel's grid
 * and byte pattern).
 *
 * None of these kernels computes anything of the attention; they exist so
 * that a roofline fraction can be read against what the chip sustains as
 * well as against its published peak.  Every buffer is a caller-owned device
 * buffer; every call enqueues on `stream` (NULL = default stream) and
 * returns 0, or a nonzero hipError_t when an argument is out of range (no
 * launch then) or the launch fails.
 */
#ifndef SDATTN_PROBES_H
#define SDATTN_PROBES_H

#ifdef __cplusplus
extern "C" {
#endif

/* Instruction-stream probe: `blocks` workgroups of eight waves (two per
 * SIMD: wave w runs on SIMD w % 4).  Waves in the MFMA role issue `it_m`
 * iterations of four independent v_mfma_f32_32x32x16_f16 (131072 flops per
 * iteration and wave); waves in the VALU role issue `it_v` iterations of 16
 * independent operations of the chosen kind (v_fma_f32 or v_exp_f32).
 *   mode 0: every wave MFMA            mode 1: every wave FMA
 *   mode 2: every wave EXP             mode 3: waves 0-3 MFMA, 4-7 FMA
 *   mode 4: waves 0-3 MFMA, 4-7 EXP    mode 5: waves 0-3 MFMA, 4-7 idle
 *   mode 6: waves 0-3 idle, 4-7 FMA    mode 7: waves 0-3 idle, 4-7 EXP
 *   mode 8: every wave MFMA on random operands (four distinct A and B
 *           operands in turn, bits that toggle like real activations; the
 *           other modes use near-constant ones)
 * out: blocks * 512 floats (a checksum per lane, keeps the streams live).
 * clk: 4 values from the first wave of workgroup 0: the shader-clock counter
 *      (s_memtime) and the constant 100 MHz counter (s_memrealtime) at the
 *      start and at the end of its stream; may be NULL.
 * Limits: 0 <= mode <= 8, 1 <= blocks <= 65536, 0 <= it_m, it_v <= 1 << 20. */
int sdattn_probe_mix(int mode, int blocks, int it_m, int it_v, float* out,
                     unsigned long long* clk, void* stream);

/* The D = 40 self-attention tile's instruction mix without its data
 * movement: `blocks` workgroups of eight waves (two per SIMD), each wave
 * `iters` iterations of two 32-query x 32-key pairs that share every operand
 * read -- K rows from a static LDS tile into 2 x 3 chained 32x32x16 MFMAs,
 * per pair 16 v_fma_f32, 16 v_exp_f32 and 8 conversions, V^T by
 * transposing LDS reads into 2 x 4 MFMAs.  mode bit 0: with the
 * exponentials; bit 1: operands of random sign and mantissa (bits that toggle
 * like real activations) instead of near-constant ones.  The second wave of
 * each SIMD (waves 4-7) starts `stagger` x 64 cycles after the first, to
 * shift the two waves' phases against each other.
 * out: blocks * 512 floats.
 * clk: 4 values from the first wave of workgroup 0, as for sdattn_probe_mix
 *      (the shader clock under this mix); may be NULL.
 * Limits: 1 <= blocks <= 65536, 1 <= iters <= 1 << 20, 0 <= mode <= 3,
 * 0 <= stagger <= 64. */
int sdattn_probe_tile(int blocks, int iters, int mode, int stagger, float* out, unsigned long long* clk,
                      void* stream);

/* dst[0 .. bytes) = src[0 .. bytes) with 16-byte loads and stores, grid-stride
 * over `blocks` workgroups of 256 threads.  bytes % 16 == 0, pointers 16-byte
 * aligned, the two ranges disjoint. */
int sdattn_probe_copy(const void* src, void* dst, long long bytes, int blocks, void* stream);

/* Reads src[0 .. bytes) with 16-byte loads (grid-stride over `blocks`
 * workgroups of 256 threads) and writes one XOR of what each thread read to
 * sink[thread] (sink holds blocks * 256 words).  bytes % 16 == 0. */
int sdattn_probe_read(const void* src, long long bytes, unsigned* sink, int blocks, void* stream);

/* The cross-attention kernel's data movement without its arithmetic: for
 * Q [B,H,Lq,D] and K, V [B,H,Lk,D] (16-bit elements, D % 8 == 0, D <= 160,
 * Lk <= 128), workgroups of `waves` waves (2, 4 or 8) each take 32 * waves
 * query rows of one (b, h) (one 32-row strip per wave, the same XCD remap of
 * the workgroup index), copy all of that head's K and V and their Q rows into
 * LDS with 16-byte direct copies, and after one barrier store the Q rows to
 * O [B,H,Lq,D] unchanged; sink receives one word per workgroup
 * (B * H * ceil(Lq / (32 * waves)) words). */
int sdattn_probe_strip_copy(const void* q, const void* k, const void* v, void* o, unsigned* sink,
                            int B, int H, int Lq, int Lk, int D, int waves, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SDATTN_PROBES_H */
