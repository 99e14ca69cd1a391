// Host-side launchers of the MPM kernels. Arguments are validated by the
// C ABI layer before any of these is called; each returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpm {

enum Dtype : int { kF32 = 0, kBf16 = 1 };

// Affinity + per-candidate-tile argmax partials: pv/pi are [B][partial_tiles(N)][N].
// start/stop (may be null) are bound to the first and last of its dispatches (hipExtLaunchKernel).
// xinv (may be null): given inverse row norms, one float per row of x (packed like x); the
// kernels then do not sum the norms themselves. Only where affinity_takes_norms(D, dt)
// (hipErrorInvalidValue otherwise).
hipError_t launch_affinity(const void* x, const int32_t* x_off, int B, int N, int D, int dt, float* pv,
                           int32_t* pi, hipStream_t stream, hipEvent_t start = nullptr, hipEvent_t stop = nullptr,
                           const float* xinv = nullptr);
// Whether launch_affinity takes given inverse norms for rows of D values of dtype dt
// (bfloat16 rows a whole number of 64 bytes: the persistent kernels).
bool affinity_takes_norms(int D, int dt);
// Partial slots per token in the workspace (the tile stride of pv/pi): ceil(N / 64).
int partial_tiles(int N);
// Candidate rows covered by one partial of the kernel launch_affinity picks for B images.
int partial_tile_width(int B, int D, int dt, int N);
// Work schedule of the persistent affinity kernel: every (query block, candidate
// tile) pair, only the pairs on and above the diagonal (the symmetric schedule),
// or a choice by batch shape. Process-wide; returns the previous mode, or -1 (and
// changes nothing) for an unknown mode.
enum AffinitySchedule : int { kScheduleAuto = 0, kScheduleFull = 1, kScheduleSymmetric = 2, kScheduleFull64 = 3 };
int set_affinity_schedule(int mode);
// The schedule (kScheduleFull, kScheduleSymmetric or kScheduleFull64) launch_affinity would run
// for this shape on the current device under the current mode.
hipError_t affinity_schedule(int B, int N, int D, int dt, int* schedule);
hipError_t launch_reduce_partials(const float* pv, const int32_t* pi, const void* x, const int32_t* x_off, int B,
                                  int N, int D, int dt, int32_t* nb, float* best, hipStream_t stream);
hipError_t launch_pair_compact_partials(const float* pv, const int32_t* pi, int T, int ct, int32_t* nb,
                                        const int32_t* x_off, int B, int N, int32_t* map, int32_t* src,
                                        int32_t* count, hipStream_t stream);

hipError_t launch_pair_compact(const int32_t* nb, const int32_t* x_off, int B, int N,
                               int32_t* map, int32_t* src, int32_t* count, hipStream_t stream);

// y_inv (may be null) receives 1 / max(||y_k||, 1e-12) of every merged row k, packed like y.
hipError_t launch_pair_average(const void* x, const int32_t* x_off, const int32_t* src,
                               const int32_t* count, int B, int N, int D, int dt, void* y,
                               int32_t* y_off, hipStream_t stream, float* y_inv = nullptr);

hipError_t launch_compose(const int32_t* map_a, const int32_t* map_b, int B, int N,
                          int32_t* map_ab, hipStream_t stream);

// map2 (may be null): gather through map2[map[i]] instead, writing that composed
// entry to map_ab (may be null) once per token.
hipError_t launch_unmerge(const void* z, const int32_t* z_off, const int32_t* map,
                          const void* z_spec, int E, int B, int N, int D, int dt, void* out,
                          hipStream_t stream, const int32_t* map2 = nullptr, int32_t* map_ab = nullptr);

}  // namespace mpm
