/*
 * wavepp_probe.h -- measurement probe of libwavepp_attn.so (not part of the attention path): the
 * dense bf16 matrix-core rate and the shader clock of the GPU it runs on, so that a roofline can be
 * quoted against what the chip actually sustains as well as against its nominal peak.
 *
 * The probe kernel keeps every operand in registers: each wave runs `iters` rounds of four
 * independent v_mfma_f32_32x32x16_bf16 chains (32 x 32 x 16 x 2 = 32,768 FLOP each), then writes
 * one float per thread to `sink` so the work is not optimized away.  Lane 0 of workgroup 0 records
 * s_memtime (shader clock cycles) and s_memrealtime (a 100 MHz counter) before and after its loop;
 * their ratio gives the shader clock while the matrix cores are busy.
 *
 * Arguments (device pointers, caller-owned):
 *   workgroups  grid size, >= 1; each workgroup is 512 threads (8 waves)
 *   iters       rounds per wave, >= 1
 *   random_operands  0: a few small constant operand values; 1: random-bit bf16 operands spread
 *               like N(0,1) samples (more bits toggle, as with attention's Q/K/V, and more power)
 *   sink        float[workgroups * 512]
 *   clocks      uint64[4]: memtime start, memrealtime start, memtime end, memrealtime end
 * FLOP per launch = workgroups * 8 * iters * 4 * 32768.
 * Errors: WAVEPP_EINVAL for a non-positive size or a NULL pointer; launch errors as WAVEPP_EHIP.
 *
 * wavepp_probe_hbm_read: the rate at which plain streaming reads move data from HBM, the practical
 * ceiling for the gather-bound waves (their K/V pages are read once, nothing comparable is written).
 * Each thread of `workgroups` x 256 reads 16-byte words of `src` grid-stride, four 4 KiB-apart words
 * per round, XORs them together and writes one uint32 to `sink`; every byte of `src` is read exactly
 * once, so the XOR of all of `sink` equals the XOR of all 32-bit words of `src`.
 *   src         device buffer, 16-byte aligned, `bytes` long (a multiple of 16), caller-owned
 *   workgroups  grid size, >= 1 (a few thousand fill the chip's memory queues)
 *   sink        device uint32[workgroups * 256], caller-owned
 * Bytes read per launch = bytes.  Errors: WAVEPP_EINVAL for a non-positive or unaligned size, an
 * unaligned or NULL pointer; launch errors as WAVEPP_EHIP.
 */
#ifndef WAVEPP_PROBE_H
#define WAVEPP_PROBE_H

#include "wavepp_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

int wavepp_probe_mfma(int32_t workgroups, int32_t iters, int32_t random_operands, float* sink,
                      unsigned long long* clocks, hipStream_t stream);
int wavepp_probe_hbm_read(const void* src, int64_t bytes, int32_t workgroups, uint32_t* sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* WAVEPP_PROBE_H */
