// Host-side launchers of the MPM kernels. Arguments are validated by the
// C ABI layer before any of these is called; each returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpm {

enum Dtype : int { kF32 = 0, kBf16 = 1 };

// Work schedule of the persistent affinity kernel (the mpm_schedule values of the C ABI).
enum AffinitySchedule : int { kScheduleAuto = 0, kScheduleFull = 1, kScheduleSymmetric = 2, kScheduleFull64 = 3 };
bool valid_schedule(int schedule);

// Affinity + per-candidate-tile argmax partials: pv/pi are [B][partial_tiles(N)][N].
// start/stop (may be null) are bound to the first and last of its dispatches (hipExtLaunchKernel).
// xinv (may be null): given inverse row norms, one float per row of x (packed like x); the
// kernels then do not sum the norms themselves. Only where affinity_takes_norms(D, dt)
// (hipErrorInvalidValue otherwise).
hipError_t launch_affinity(const void* x, const int32_t* x_off, int B, int N, int D, int dt, int schedule, float* pv,
                           int32_t* pi, hipStream_t stream, hipEvent_t start, hipEvent_t stop, const float* xinv);
// Whether launch_affinity takes given inverse norms for rows of D values of dtype dt
// (bfloat16 rows a whole number of 64 bytes: the persistent kernels).
bool affinity_takes_norms(int D, int dt);
// Partial slots per token in the workspace (the tile stride of pv/pi): ceil(N / 64).
int partial_tiles(int N);
// Candidate rows covered by one partial of the kernel launch_affinity picks for this call.
int partial_tile_width(int B, int D, int dt, int N, int schedule);
// ... and of launch_affinity_local's kernel: the rows of its square blocks on the
// persistent kernel's symmetric schedule (`requested`, 128 or 256; 0: whichever an
// estimate of the launch on a full raster grid of grid_w columns finds faster on the
// current device), else N (one slot covering the image).
int local_block_rows(int B, int N, int D, int dt, int grid_w, int radius, int requested);
bool valid_local_block_rows(int requested);
// The schedule (kScheduleFull, kScheduleSymmetric or kScheduleFull64) launch_affinity runs
// for this shape and requested schedule on the current device.
hipError_t affinity_schedule(int B, int N, int D, int dt, int schedule, int* used);

hipError_t launch_reduce_partials(const float* pv, const int32_t* pi, int ct, const void* x, const int32_t* x_off,
                                  int B, int N, int D, int dt, int32_t* nb, float* best, hipStream_t stream);
// Compaction (map, src, offsets) from the partials (reduced first) or from nb. sync (may be
// null): the workspace's arrival counters, zero on entry and exit; with them the last
// image's workgroup scans the offsets, without them a second launch does.
hipError_t launch_pair_compact_partials(const float* pv, const int32_t* pi, int T, int ct, int32_t* nb,
                                        const int32_t* x_off, int B, int N, int32_t* map, int32_t* src,
                                        int32_t* y_off, int32_t* sync, hipStream_t stream);
hipError_t launch_pair_compact(const int32_t* nb, const int32_t* x_off, int B, int N, int32_t* map, int32_t* src,
                               int32_t* y_off, int32_t* sync, hipStream_t stream);
hipError_t launch_zero_words(int32_t* p, long words, hipStream_t stream);

// y_inv (may be null) receives 1 / max(||y_k||, 1e-12) of every merged row k, packed like y.
// y_pos (may be null) receives each merged row's grid position: its
// representative's pos (packed like x; null: its index in the image).
hipError_t launch_pair_average(const void* x, const int32_t* x_off, const int32_t* src, const int32_t* y_off, int B,
                               int N, int D, int dt, void* y, float* y_inv, hipStream_t stream,
                               const int32_t* pos = nullptr, int32_t* y_pos = nullptr);
// The affinity partials under the locality constraint (Sec. 5): candidates of each token
// restricted to the cells within `radius` rows and columns of its own on a grid of
// grid_w columns (pos: raster positions packed like x, or null for each token's index;
// xinv: given inverse norms, or null to sum them); partials of
// local_block_rows(B, N, D, dt, grid_w, radius, block_rows) candidate rows each, every
// slot of an image's tiles written (-inf, -1 where the window reaches no candidate of a tile).
hipError_t launch_affinity_local(const void* x, const int32_t* x_off, const float* xinv, const int32_t* pos,
                                 int grid_w, int radius, int block_rows,
                                 int B, int N, int D, int dt, float* pv, int32_t* pi, hipStream_t stream,
                                 hipEvent_t start, hipEvent_t stop);

// Padded batch layout: packed rows (offsets z_off) to [B][P] rows of rowbytes bytes, zero
// rows past each image (unpad = false), or back to the packed layout (unpad = true).
hipError_t launch_pad(const void* z, const int32_t* z_off, int B, int P, long rowbytes, void* out, bool unpad,
                      hipStream_t stream);

hipError_t launch_compose(const int32_t* map_a, const int32_t* map_b, int B, int N,
                          int32_t* map_ab, hipStream_t stream);

// map2 (may be null): gather through map2[map[i]] instead, writing that composed
// entry to map_ab (may be null) once per token.
hipError_t launch_unmerge(const void* z, const int32_t* z_off, const int32_t* map,
                          const void* z_spec, int E, int B, int N, int D, int dt, void* out,
                          hipStream_t stream, const int32_t* map2 = nullptr, int32_t* map_ab = nullptr);

// Checked mode: validation of caller data on the device. Each launcher ORs its bit into
// *verdict (a device word the caller cleared) when a precondition fails.
enum CheckBit : int32_t { kCheckOffsets = 1, kCheckValues = 2, kCheckPositions = 4 };
// Packed offsets: off[0] >= 0, lo_n <= off[b+1] - off[b] <= N, off[B] <= cap (cap >= 0);
// with `within` (may be null), also at most the count within[b+1] - within[b].
hipError_t launch_check_offsets(const int32_t* off, int B, int N, int lo_n, long cap, const int32_t* within,
                                int32_t* verdict, hipStream_t stream);
// Slot values v[(b*N + i)*per + e] for i below the count of cnt_off (null: N): each in
// [lo, count of hi_off) (hi_off null: N); `bit` on failure.
hipError_t launch_check_slots(const int32_t* v, int per, const int32_t* cnt_off, int lo, const int32_t* hi_off, int B,
                              int N, int32_t bit, int32_t* verdict, hipStream_t stream);
// Neighbours: nb in [0, n_b) and not the token itself, -1 for a one-token image.
hipError_t launch_check_nb(const int32_t* nb, const int32_t* x_off, int B, int N, int32_t* verdict, hipStream_t stream);
// Grid positions: in [0, limit) and non-decreasing in row (pos / grid_w) along each image.
hipError_t launch_check_pos(const int32_t* pos, const int32_t* x_off, int B, int N, int grid_w, long limit,
                            int32_t* verdict, hipStream_t stream);
// Given inverse norms: finite and positive.
hipError_t launch_check_inv(const float* inv, const int32_t* x_off, int B, int N, int32_t* verdict,
                            hipStream_t stream);
// Token values: finite.
hipError_t launch_check_finite(const void* x, const int32_t* x_off, int B, int N, int D, int dt, int32_t* verdict,
                               hipStream_t stream);

}  // namespace mpm
