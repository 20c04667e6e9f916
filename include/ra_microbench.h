/* Hardware ceilings for the rollout-attention kernels, measured on the GPU
 * they run on: matrix-core rate of the bf16 product the append kernel uses
 * (with the shader clock it ran at), LDS read bandwidth per compute unit,
 * and HBM read rate of a streaming and of a paged (shuffled 4 KiB blocks)
 * access pattern. These are the "achievable" figures the benchmark reports
 * beside the vendor peaks; they compute nothing of the attention itself.
 *
 * Built as libra_microbench.so beside librollout_attn.so. Plain device
 * pointers, asynchronous on `stream`; every function returns 0 on success,
 * 1 for a null pointer, 2 for a bad size and 5 when the launch fails. The
 * caller owns every buffer; the library allocates nothing.
 */
#ifndef RA_MICROBENCH_H
#define RA_MICROBENCH_H

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Threads of one workgroup of ra_mb_mfma_bf16 (4 waves, one per SIMD when a
 * compute unit holds one workgroup). */
#define RA_MB_MFMA_THREADS 256
/* bf16 operand elements ra_mb_mfma_bf16 reads: 8 operands of 8 elements per
 * thread (4 A and 4 B registers of v_mfma_f32_32x32x16_bf16). */
#define RA_MB_MFMA_OPERANDS (RA_MB_MFMA_THREADS * 64)
/* Threads of one workgroup of ra_mb_lds_read. */
#define RA_MB_LDS_THREADS 512

/* Each wave runs `iters` rounds of 4 independent v_mfma_f32_32x32x16_bf16
 * products (32768 flops each) on the operands given (bf16, RA_MB_MFMA_OPERANDS
 * elements, device memory; pass random values for the rate on attention-like
 * data, zeros for the data-independent rate). Work = blocks * 4 waves * iters
 * * 4 * 32768 flops. sink: fp32 [blocks * 256] (sums of the accumulators, so
 * that nothing is optimised away). clocks: int64 [4], written by the first
 * wave: shader-clock counter (s_memtime) and 100 MHz real-time counter
 * (s_memrealtime) before and after its loop; their ratio gives the shader
 * clock while the products ran. */
int ra_mb_mfma_bf16(const void *operands, int32_t blocks, int32_t iters, float *sink,
                    int64_t *clocks, hipStream_t stream);

/* Each of blocks * RA_MB_LDS_THREADS threads reads 8 x 16 bytes of LDS per
 * round (ds_read_b128, consecutive lanes on consecutive 16-byte words: no bank
 * conflicts) for `iters` rounds. Bytes read = blocks * 512 * iters * 128.
 * sink: uint32 [blocks * 512]; clocks as for ra_mb_mfma_bf16. */
int ra_mb_lds_read(int32_t blocks, int32_t iters, uint32_t *sink, int64_t *clocks,
                   hipStream_t stream);

/* Reads `bytes` (a multiple of 4096) from src once, 16 bytes per lane: each
 * workgroup of 256 threads reads four 4 KiB blocks per round (four loads per
 * lane in flight), the workgroups of a round taking consecutive block numbers.
 * With order == NULL block number j is block j (address order); otherwise it
 * is block order[j] (int32 [bytes / 4096], device memory, values clamped to
 * the buffer), the access pattern of a paged cache with shuffled pages.
 * sink: uint32 [blocks * 256]. */
int ra_mb_stream_read(const void *src, int64_t bytes, const int32_t *order, int32_t blocks,
                      uint32_t *sink, hipStream_t stream);

/* Reads `bytes` from src once in shuffled blocks of block_bytes (1024, 2048 or
 * 4096; bytes / block_bytes a power of two, at least 16): block j of the pass
 * is block mix(j) of src for a fixed bijection mix (no block numbers are read
 * from memory), 16 bytes per lane, four loads per lane in flight, one load
 * instruction of a 256-thread workgroup taking 4096 / block_bytes blocks. The
 * read rate of a paged pool as a function of its block size. sink: uint32
 * [blocks * 256]. */
int ra_mb_block_read(const void *src, int64_t bytes, int32_t block_bytes, int32_t blocks,
                     uint32_t *sink, hipStream_t stream);

/* Reads an L2-resident buffer (bytes: a power of two from 64 KiB to 16 MiB,
 * small enough to stay in each XCD's 4 MiB L2 when at most 2 MiB) over and
 * over: each of blocks workgroups of 256 threads runs `iters` rounds in which
 * every wave issues 16 load instructions of 1 KiB (16 bytes per lane),
 * walking the buffer from a per-workgroup offset. to_lds != 0: direct
 * global-to-LDS loads (global_load_lds_dwordx4, 64 KiB of LDS per
 * workgroup); otherwise loads into registers. Bytes moved = blocks * iters *
 * 64 KiB (the register form reads 8 KiB more per wave). The rate at which the
 * L2 feeds the compute units. sink: uint32 [blocks * 256]. Returns 1 for a
 * null pointer, 2 for a bad size (or iters outside [1, 2^24]). */
int ra_mb_l2_read(const void *src, int64_t bytes, int32_t to_lds, int32_t blocks, int32_t iters,
                  uint32_t *sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* RA_MICROBENCH_H */
