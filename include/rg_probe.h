/*
 * rg_probe.h -- a read-bandwidth probe for librg's measurements (librg_probe.so).
 *
 * The linear layer at batch 1 is bound by reading the weights from HBM.  This
 * library holds one kernel that reads a buffer and does nothing else, in the
 * access pattern that measured fastest on MI355X (every wave reads whole 8 KB
 * pieces with 16-byte vector loads, consecutive pieces on consecutive waves, so
 * that at any moment the grid reads one compact window of memory).  Its time
 * over a layer's weight bytes is the floor the layer's kernels are held against
 * (the benchmark's --floors mode).  It is not part of the product path.
 *
 *   src    device pointer, 16-byte aligned; bytes a multiple of 8192, >= 8192
 *   sink   device pointer to one uint32 per launched thread (grid * 256), written
 *          with the XOR of the words the thread read (keeps the loads alive)
 *   grid   workgroups of 256 threads, 1 .. 65536
 * Returns 0, 1 on an invalid argument, 4 on a launch error.
 */
#ifndef RG_PROBE_H
#define RG_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int rg_probe_read(const void* src, int64_t bytes, uint32_t* sink, int32_t grid, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RG_PROBE_H */
