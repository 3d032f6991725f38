// Launchers of kernels defined in graph.hip and used by the step driver.
#pragma once

#include "common.h"

namespace janus {

// Bit 1: bad offsets; bit 2 (only when rc > 0): cell not diagonal-positive or far smaller than rc.
void launch_validate_struct(hipStream_t st, const int* offsets, int S, int N, const float* cell, float rc,
                            int* flag);
void launch_atom_struct(hipStream_t st, const int* offsets, int S, int N, int* sid);
// Exclusive scan of n ints into out[0..n] (out[n] = total); when the total
// overflows int32, flag |= 16 (bit 4).  scratch holds scan_scratch_bytes(n) bytes.
size_t scan_scratch_bytes(long long n);
void launch_exclusive_scan(hipStream_t st, const int* in, int n, int* out, int* flag, long long* scratch);
// geo[e] = (u_x, u_y, u_z, r); B, dB [Ne, nb].  With rc3 > 0 also the
// three-body basis B3, dB3 [Ne, nb] and envelope u3, du3 [Ne] at cutoff rc3;
// with d2B the second radial derivative of the basis [Ne, nb].
void launch_geometry(hipStream_t st, const float* pos, const float* cell, const int* sid, const int* ei,
                     const int* ej, const int8_t* shift, int Ne, float rc, int nb, float4* geo, float* B,
                     float* dB, float rc3 = 0.f, float* B3 = nullptr, float* dB3 = nullptr, float* u3 = nullptr,
                     float* du3 = nullptr, float* d2B = nullptr);

}  // namespace janus
