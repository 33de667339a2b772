/*
 * rg_probe.h -- a read-bandwidth probe for librg's measurements (librg_probe.so).
 *
 * The linear layer at batch 1 is bound by reading the weights from HBM.  This
 * library holds one kernel that reads a buffer and does nothing else, in the
 * access pattern that measured fastest on MI355X (every wave reads whole 8 KB
 * pieces with 16-byte non-temporal vector loads, consecutive pieces on
 * consecutive waves, so that at any moment the grid reads one compact window
 * of memory).  Its time
 * over a layer's weight bytes is the floor the layer's kernels are held against
 * (the benchmark's --floors mode).  It is not part of the product path.
 *
 *   src    device pointer, 16-byte aligned; bytes a multiple of 8192, >= 8192
 *   sink   device pointer to one uint32 per launched thread (grid * 256), written
 *          with the XOR of the words the thread read (keeps the loads alive)
 *   grid   workgroups of 256 threads, 1 .. 65536
 * Returns 0, 1 on an invalid argument, 4 on a launch error.
 *
 * rg_probe_fma: the binary32 FMA issue rate the kernels can reach, for the
 * ceilings they are held against.  Every thread of grid workgroups of 256 runs
 * `chains` (8 or 16) independent v_fmac_f32 chains for iters * 64 steps, each
 * FMA's first operand read plainly (mode 0), through a DPP row broadcast
 * (mode 1), through a DPP quad broadcast (mode 2), from an SGPR shared by the
 * wave (mode 3), or from an SGPR and a plain VGPR in turn (mode 4), the forms
 * the kernels use; 2 * 64 *
 * iters * grid * 256 flops per launch.  out: device pointer to grid * 256
 * floats (the chains' sums).  Returns 0, 1 on an invalid argument, 4 on a
 * launch error.
 */
#ifndef RG_PROBE_H
#define RG_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int rg_probe_read(const void* src, int64_t bytes, uint32_t* sink, int32_t grid, void* stream);
int rg_probe_fma(int32_t mode, int32_t chains, float* out, int32_t grid, int32_t iters, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RG_PROBE_H */
