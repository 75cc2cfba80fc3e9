/* libshardprobe.so: measurement aids beside the shard path (not part of it).
 *
 * The shard convolution's bf16 MFMA rate is reported against the part's
 * published dense peak. A kernel that does nothing but matrix instructions
 * shows what the part sustains at its own clock under that load; the entry
 * point below runs such a kernel so that a benchmark can print the measured
 * ceiling next to the published one. */
#ifndef SHARDPROBE_H
#define SHARDPROBE_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Launches `blocks` workgroups of 4 waves. Each wave runs 4 independent
 * accumulation chains of v_mfma_f32_32x32x16_bf16, `iters` instructions per
 * chain: 2*32*32*16 * 4 * iters flops per wave, 4 waves per block.
 *   random: 0 = constant operands (small values, few toggling bits);
 *           1 = roughly N(0, 1) bf16 operands, 4 A and 4 B fragments per lane
 *               in rotation, so that the operands change from one instruction
 *               to the next as they do in a convolution;
 *   out: device memory, blocks*256 floats, written (the accumulated sums, so
 *        the work is not optimised away);
 *   clk: device memory, 2*blocks uint64, written: for wave 0 of block b,
 *        clk[2b] = shader-clock ticks and clk[2b+1] = 100 MHz reference ticks
 *        between the first and the last instruction (their ratio is the
 *        shader clock).
 * Asynchronous on `stream`; the caller owns every buffer. Returns 0; 1 for
 * iters < 1 or not a multiple of 4, blocks < 1 or a null buffer (nothing
 * launched); 3 when the launch fails. */
int shard_probe_mfma_bf16(int64_t iters, int32_t blocks, int32_t random, float* out, uint64_t* clk,
                          hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif
