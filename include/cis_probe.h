/*
 * cis_probe.h — bandwidth probes used to measure the roofline of the CIS row kernel
 * (libcis_probe.so). Not part of the loss; a measurement helper for benchmarks.
 */
#ifndef CIS_PROBE_H
#define CIS_PROBE_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * cis_probe_bandwidth — streams `rows` rows of `row_bytes` bytes with the row kernel's access
 * pattern (one 1024-thread workgroup per row at a time, 16-byte non-temporal buffer accesses,
 * the whole row in flight, rows after a workgroup's first taken from a queue as the fused pass
 * takes them) on `stream`, without synchronising.
 *
 *   mode 0: copy src -> dst; 1: read src only; 2: write dst only
 *   mode 3: copy src -> dst of rows*row_bytes contiguous bytes with short-lived 128-thread
 *           workgroups of 4 KiB each (two 16-byte non-temporal vectors per thread): the
 *           fastest equal read/write stream found on this part (grid is ignored, row_bytes
 *           only needs to be a multiple of 16)
 *   mode 4: read src only, in the workgroups of mode 3: the fastest read stream found
 *   src, dst   device buffers of rows*row_bytes bytes (src unused in mode 2, dst in modes 1, 4)
 *   row_bytes  multiple of 16, at most 19*1024*16
 *   grid       workgroups (persistent over rows), >= 1
 *   sink       device uint32[1026], 8-byte aligned: words 0..1023 receive nothing in practice
 *              (the read modes keep their loads alive through them), words 1024..1025 hold
 *              the row queue's counter of modes 0-2, which the call clears with a kernel of
 *              its own first; required in modes 0, 1, 2 and 4
 * Returns 0, or -1 (NULL pointer), -2 (row_bytes, a misaligned sink, or a mode-3/4 size beyond
 * 2^31 workgroups), -4 (mode/rows/grid), -6 (launch failed).
 */
int cis_probe_bandwidth(int mode, const void* src, void* dst, int64_t rows, int64_t row_bytes,
                        int grid, uint32_t* sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* CIS_PROBE_H */
