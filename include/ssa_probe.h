/*
 * ssa_probe.h -- measurement support: the achievable peaks of the GPU that
 * the rooflines of the library's kernels are stated against, next to the
 * published ones.  Not part of any serving path.
 *
 * Same conventions as ssa.h: 0 or a negative SSA_ERR_* code, validation before
 * any HIP call, no allocation.
 */
#ifndef SSA_PROBE_H
#define SSA_PROBE_H

#include <stddef.h>
#include <stdint.h>

#include "ssa.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Streams `bytes` of device memory at `src` (16-byte aligned, bytes a multiple
 * of 16 and > 0) through 16-byte vector loads, several in flight per thread,
 * and writes one 32-bit XOR of the data per workgroup to out[workgroups]
 * (`workgroups` in 1..65536) so that no load can be dropped.  Bytes read per
 * launch: `bytes`.
 * Errors: SSA_ERR_ARG, SSA_ERR_NULL, SSA_ERR_HIP.
 */
int ssa_probe_hbm_read(const void* src, size_t bytes, uint32_t* out, int32_t workgroups,
                       void* stream);

/*
 * Gathers whole chunks of `chunk_bytes` (1024, 2048, 4096, 8192 or 16384) from
 * the device buffer `src` (`src_bytes` long, 16-byte aligned, at least one
 * chunk): chunk i of the launch is the one at byte chunk_index[i] * chunk_bytes
 * (chunk_index: n_chunks >= 1 int32 in device memory, read in order; an index
 * outside [0, src_bytes / chunk_bytes) is clamped into it).  Each wave keeps
 * 16 KB of 16-byte loads in flight, whole chunks at a time, the pattern of the
 * attention kernel's decode reads (4 KB of one page and kv head per load
 * group).  `pattern` 0: each 16-byte load instruction of a wave reads one whole
 * 1 KB row of the chunk; 1 (4 KB chunks only): it reads 64 B of each of 16
 * rows of 256 B, the key rows' pattern of the attention kernel's decode loads.
 * Writes one 32-bit XOR of the data per workgroup to out[workgroups]
 * (`workgroups` in 1..65536).  Bytes read per launch: n_chunks * chunk_bytes,
 * plus re-reads of the last chunk that fill the final step of each wave.
 * Errors: SSA_ERR_ARG, SSA_ERR_NULL, SSA_ERR_HIP.
 */
int ssa_probe_hbm_gather(const void* src, size_t src_bytes, const int32_t* chunk_index,
                         int32_t n_chunks, int32_t chunk_bytes, int32_t pattern, uint32_t* out,
                         int32_t workgroups, void* stream);

/*
 * Runs `iters` rounds of 16 independent v_mfma_f32_16x16x32_bf16 chains in
 * each wave of `workgroups` workgroups of 256 threads (iters in 1..2^20,
 * workgroups in 1..65536) on register data, and writes one float per
 * workgroup to out[workgroups].  Flops per launch:
 * workgroups * 4 * iters * 16 * 16384.
 * Errors: SSA_ERR_ARG, SSA_ERR_NULL, SSA_ERR_HIP.
 */
int ssa_probe_mfma_bf16(int32_t iters, int32_t workgroups, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SSA_PROBE_H */
