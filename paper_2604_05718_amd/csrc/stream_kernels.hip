// HBM-streaming steps of MPM for gfx950: cluster means (Eq. 2), map
// composition (Eq. 3) and gather reconstruction (Eq. 4).
//
// The row kernels treat a token row as D*s/16 independent 16-byte vectors and
// deal them to the lanes with the workgroup size as stride, so any D keeps all
// lanes busy and every global access is a 16-byte, fully coalesced load or
// store. A lane loads a small batch of vectors before storing any, so several
// loads per lane are in flight (one load then one store per lane left the
// gather latency-bound). The merged rows of the pair average are stored plainly:
// the next insertion's affinity and average, or the gather, read them right
// after, and a plain store leaves them in the last-level cache. The gather's
// full token grid is read by nothing after it and is stored with non-temporal
// hints.
#include "mpm_device.h"
#include "mpm_launch.h"

namespace mpm {
namespace {

constexpr int kRowThreads = 256;
constexpr int kRowBytesPerBlock = 8192;      // output bytes one workgroup handles
constexpr int kGatherBytesPerBlock = 16384;  // ... in the gather, which first resolves its rows' sources
// Vectors each thread loads before storing them (loads in flight per thread).
constexpr int kGatherBatch = 4;
constexpr int kAverageBatch = 2;  // each vector of the average already loads two rows
constexpr int kMaxRowsPerBlock = 4096;       // rows one gather workgroup resolves into LDS (16 KB)
constexpr int kInvBatch = 8;  // vectors per lane at most, in the pair average that also writes row norms
constexpr int kXcdCount = 8;                    // MI355X: workgroups are dealt round-robin to 8 XCDs
constexpr long kXcdL2Bytes = 4L << 20;          // ... each with a 4 MB L2

// Lanes per row in the pair average that also writes row norms: a power of two, at
// most a wave, enough for at most kInvBatch vectors per lane where a wave allows it.
__host__ __device__ constexpr int inv_lanes(int vpr)
{
    int g = 1;
    while (g < kWave && g * kInvBatch < vpr) g *= 2;
    return g;
}

// Walks the flat range [f0, f1) of 16-byte vectors of a row-major block whose rows
// hold `vpr` vectors, U vectors per lane at a time (stride of the workgroup size):
// load(row, vec) for all U, then store(row, vec, value) for all U. Row and column
// advance incrementally (no per-element division).
template <int U, class Load, class Store>
__device__ __forceinline__ void for_each_vec_batched(long f0, long f1, int vpr, Load load, Store store)
{
    const int t = threadIdx.x;
    long f = f0 + t;
    if (f >= f1) return;
    long row = f / vpr;
    int col = (int)(f - row * vpr);
    const int step_rows = kRowThreads / vpr;
    const int step_cols = kRowThreads - step_rows * vpr;
    while (f < f1) {
        u32x4 v[U];
        long rr[U];
        int cc[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            ok[u] = f < f1;
            rr[u] = row;
            cc[u] = col;
            if (ok[u]) v[u] = load(row, col);
            f += kRowThreads;
            row += step_rows;
            col += step_cols;
            if (col >= vpr) {
                col -= vpr;
                row += 1;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) store(rr[u], cc[u], v[u]);
    }
}

// Output rows of image b in a packed buffer of capacity B*N rows, from offsets that
// the compaction wrote. The clamps change nothing for offsets that follow the
// contract (0 <= count <= N, monotone, within capacity); they keep a kernel in
// bounds if an upstream fault ever left them unwritten.
struct Span {
    int off, cnt;
};
__device__ __forceinline__ Span output_span(const int32_t* y_off, int b, int N, int B)
{
    const int o = y_off[b];
    const int c = min(max(y_off[b + 1] - o, 0), N);
    const long cap = (long)B * N;
    return Span{(int)min(max((long)o, 0L), cap - c), c};
}
// A source row index from src, kept inside the image's n rows (same contract note).
__device__ __forceinline__ int clamp_row(int r, int n) { return min(max(r, 0), n - 1); }

// Sum of squares of the values of one 16-byte vector, in float32.
__device__ __forceinline__ float vec_sumsq(u32x4 v, Bf16)
{
    // One v_dot2c_f32_bf16 per pair of values; the words are scalars before the bit cast.
    const uint32_t w0 = v.x, w1 = v.y, w2 = v.z, w3 = v.w;
    float s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w0), __builtin_bit_cast(bf16x2, w0), 0.0f, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w1), __builtin_bit_cast(bf16x2, w1), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w2), __builtin_bit_cast(bf16x2, w2), s, false);
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w3), __builtin_bit_cast(bf16x2, w3), s, false);
}

__device__ __forceinline__ float vec_sumsq(u32x4 v, F32)
{
    float s = 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) s = fmaf(__uint_as_float(v[e]), __uint_as_float(v[e]), s);
    return s;
}

template <class S>
__global__ __launch_bounds__(kRowThreads) void pair_average_kernel(
    const uint8_t* __restrict__ x, const int32_t* __restrict__ x_off, const int32_t* __restrict__ src,
    const int32_t* __restrict__ y_off, int N, int D, int rows_per_block, uint8_t* __restrict__ y,
    const int32_t* __restrict__ pos, int32_t* __restrict__ y_pos)
{
    const int b = blockIdx.y;
    const Span sp = output_span(y_off, b, N, gridDim.y);
    const int k0 = blockIdx.x * rows_per_block;
    const int k1 = min(sp.cnt, k0 + rows_per_block);
    if (k0 >= k1) return;
    const long rowbytes = (long)D * S::kBytes;
    const int vpr = (int)(rowbytes / 16);
    const int nx = x_off ? x_off[b + 1] - x_off[b] : N;
    const uint8_t* ximg = x + (long)(x_off ? x_off[b] : b * N) * rowbytes;
    uint8_t* yimg = y + (long)sp.off * rowbytes;
    const int32_t* srcb = src + 2L * b * N;
    for_each_vec_batched<kAverageBatch>((long)k0 * vpr, (long)k1 * vpr, vpr,
        [&](long k, int c) {
            const int ia = clamp_row(srcb[2 * k], nx);
            const int ib = clamp_row(srcb[2 * k + 1], nx);
            const u32x4 va = load16(ximg + ia * rowbytes + c * 16);
            u32x4 out = va;  // a singleton is copied bit for bit
            if (ib != ia) out = mean16(va, load16(ximg + ib * rowbytes + c * 16), S{});
            return out;
        },
        [&](long k, int c, u32x4 out) { store16(yimg + k * rowbytes + c * 16, out); });
    if (y_pos) {  // grid positions of the merged rows (locality constraint): the representative's
        const int32_t* posb = pos ? pos + (x_off ? x_off[b] : b * N) : nullptr;
        for (int k = k0 + (int)threadIdx.x; k < k1; k += kRowThreads) {
            const int rep = clamp_row(srcb[2 * k], nx);
            y_pos[sp.off + k] = posb ? posb[rep] : rep;
        }
    }
}

// The pair average that also writes the inverse norm of every merged row, from the
// stored values. A group of G = inv_lanes(vpr) lanes takes a row: lane j its vectors
// j, j + G, ..., kInvBatch at a time (all loaded before any is stored), summing their
// squares in that order; a butterfly across the group adds the lanes' sums. The order
// is fixed, so the result is the same on every run. The merged rows (and positions) are
// those of pair_average_kernel, bit for bit.
template <class S>
__global__ __launch_bounds__(kRowThreads) void pair_average_inv_kernel(
    const uint8_t* __restrict__ x, const int32_t* __restrict__ x_off, const int32_t* __restrict__ src,
    const int32_t* __restrict__ y_off, int N, int D, uint8_t* __restrict__ y, float* __restrict__ y_inv,
    const int32_t* __restrict__ pos, int32_t* __restrict__ y_pos)
{
    const int b = blockIdx.y;
    const Span sp = output_span(y_off, b, N, gridDim.y);
    const int off = sp.off, cnt = sp.cnt;
    const long rowbytes = (long)D * S::kBytes;
    const int vpr = (int)(rowbytes / 16);
    const int G = inv_lanes(vpr);
    const int k0 = blockIdx.x * (kRowThreads / G);
    if (k0 >= cnt) return;
    const int k = k0 + (int)threadIdx.x / G;  // this group's row
    const int j = threadIdx.x % G;
    const bool live = k < cnt;
    const int nx = x_off ? x_off[b + 1] - x_off[b] : N;
    const uint8_t* ximg = x + (long)(x_off ? x_off[b] : b * N) * rowbytes;
    int ia = 0, ib = 0;
    if (live) {
        ia = clamp_row(src[2L * b * N + 2 * k], nx);
        ib = clamp_row(src[2L * b * N + 2 * k + 1], nx);
    }
    const uint8_t* xa = ximg + (long)ia * rowbytes;
    const uint8_t* xb = ximg + (long)ib * rowbytes;
    uint8_t* yr = y + (long)(off + k) * rowbytes;
    float t = 0.0f;
    for (int c0 = j; c0 < vpr; c0 += G * kInvBatch) {
        u32x4 v[kInvBatch];
#pragma unroll
        for (int u = 0; u < kInvBatch; ++u) {
            const int c = c0 + u * G;
            if (live && c < vpr) {
                const u32x4 va = load16(xa + c * 16);
                v[u] = va;  // a singleton is copied bit for bit
                if (ib != ia) v[u] = mean16(va, load16(xb + c * 16), S{});
            }
        }
#pragma unroll
        for (int u = 0; u < kInvBatch; ++u) {
            const int c = c0 + u * G;
            if (live && c < vpr) {
                store16(yr + c * 16, v[u]);
                t += vec_sumsq(v[u], S{});
            }
        }
    }
    for (int o = G / 2; o > 0; o >>= 1) t += __shfl_xor(t, o);
    if (live && j == 0) {
        y_inv[off + k] = 1.0f / fmaxf(sqrtf(t), 1e-12f);
        if (y_pos) y_pos[off + k] = pos ? pos[(x_off ? x_off[b] : b * N) + ia] : ia;  // the representative's
    }
}

__global__ __launch_bounds__(kRowThreads) void compose_kernel(const int32_t* map_a,
                                                              const int32_t* __restrict__ map_b, int N,
                                                              long total, int32_t* map_ab)
{
    const long t = (long)blockIdx.x * kRowThreads + threadIdx.x;
    if (t >= total) return;
    const long b = t / N;
    const int a = map_a[t];
    map_ab[t] = a < 0 ? -1 : map_b[b * N + a];
}

// Gather reconstruction. With map2 != nullptr the source of token i is the
// composition map2[map[i]] (Eq. 3 folded into Eq. 4), and map_ab (if given)
// receives that composed entry. The workgroup first resolves the source row of
// each of its output rows into LDS (one map lookup per row, not per vector),
// then streams the rows' 16-byte vectors.
template <class S>
__global__ __launch_bounds__(kRowThreads) void unmerge_kernel(
    const uint8_t* __restrict__ z, const int32_t* __restrict__ z_off, const int32_t* __restrict__ map,
    const int32_t* __restrict__ map2, int32_t* __restrict__ map_ab, const uint8_t* __restrict__ z_spec, int E,
    int N, int D, int rows_per_block, uint8_t* __restrict__ out, int B, int xcd_major)
{
    __shared__ int32_t src_row[kMaxRowsPerBlock];
    // Row block and image of this workgroup: (blockIdx.x, blockIdx.y), or, XCD-major (a
    // one-dimensional grid; workgroup L runs on XCD L % 8), every row block of an image on
    // one XCD, so the merged rows two row blocks share (a pair's tokens a grid row apart)
    // are read through one L2.
    int b = blockIdx.y, xb = blockIdx.x;
    if (xcd_major) {
        const int nx = (E + N + rows_per_block - 1) / rows_per_block;
        const int k = blockIdx.x / kXcdCount;
        b = blockIdx.x % kXcdCount + kXcdCount * (k / nx);
        xb = k % nx;
        if (b >= B) return;
    }
    const int rows = E + N;
    const int r0 = xb * rows_per_block;
    const int r1 = min(rows, r0 + rows_per_block);
    if (r0 >= r1) return;
    const long rowbytes = (long)D * S::kBytes;
    const int vpr = (int)(rowbytes / 16);
    const uint8_t* zimg = z + (long)(z_off ? z_off[b] : b * N) * rowbytes;
    const int nz = z_off ? z_off[b + 1] - z_off[b] : N;  // rows of z for image b: a map entry past them reads zeros
    const int32_t* mapb = map + (long)b * N;
    const int32_t* map2b = map2 ? map2 + (long)b * N : nullptr;
    uint8_t* oimg = out + (long)b * rows * rowbytes;
    for (int r = r0 + (int)threadIdx.x; r < r1; r += kRowThreads) {
        int m = -1;  // special rows are not looked up
        if (r >= E) {
            m = mapb[r - E];
            if (map2b) {
                m = m < 0 ? -1 : map2b[m];
                if (map_ab) map_ab[(long)b * N + r - E] = m;
            }
        }
        src_row[r - r0] = m < nz ? m : -1;
    }
    __syncthreads();
    for_each_vec_batched<kGatherBatch>((long)r0 * vpr, (long)r1 * vpr, vpr,
        [&](long r, int c) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if (r < E) {
                v = load16(z_spec + ((long)b * E + r) * rowbytes + c * 16);
            } else {
                const int m = src_row[r - r0];
                if (m >= 0) v = load16(zimg + m * rowbytes + c * 16);
            }
            return v;
        },
        [&](long r, int c, u32x4 v) { store16_stream(oimg + r * rowbytes + c * 16, v); });
}

// Padded batch layout: out[b][k] = z[z_off[b] + k] for k < n_b, zeros for n_b <= k < P
// (P = padded rows per image), one 16-byte vector per lane and step; with UNPAD the
// copy goes back, out packed from a padded z, rows k >= n_b not read.
template <bool UNPAD>
__global__ __launch_bounds__(kRowThreads) void pad_kernel(const uint8_t* __restrict__ z,
                                                          const int32_t* __restrict__ z_off, int P, long rowbytes,
                                                          int rows_per_block, uint8_t* __restrict__ out)
{
    const int b = blockIdx.y;
    const int o = z_off[b];
    const int n = min(max(z_off[b + 1] - o, 0), P);
    const int r0 = blockIdx.x * rows_per_block;
    const int r1 = min(UNPAD ? n : P, r0 + rows_per_block);
    if (r0 >= r1) return;
    const int vpr = (int)(rowbytes / 16);
    const uint8_t* packed_z = z + (long)o * rowbytes;          // pad: the image's packed rows
    const uint8_t* padded_z = z + (long)b * P * rowbytes;      // unpad: the image's padded rows
    uint8_t* padded_out = out + (long)b * P * rowbytes;
    uint8_t* packed_out = out + (long)o * rowbytes;
    for_each_vec_batched<kGatherBatch>((long)r0 * vpr, (long)r1 * vpr, vpr,
        [&](long r, int c) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if (UNPAD) v = load16(padded_z + r * rowbytes + c * 16);
            else if (r < n) v = load16(packed_z + r * rowbytes + c * 16);
            return v;
        },
        [&](long r, int c, u32x4 v) {
            if (UNPAD) store16(packed_out + r * rowbytes + c * 16, v);
            else store16(padded_out + r * rowbytes + c * 16, v);
        });
}

int rows_per_block_for(long rowbytes, long block_bytes = kRowBytesPerBlock)
{
    const long r = block_bytes / rowbytes;
    return r < 1 ? 1 : (r > kMaxRowsPerBlock ? kMaxRowsPerBlock : (int)r);
}

}  // namespace

hipError_t launch_pair_average(const void* x, const int32_t* x_off, const int32_t* src, const int32_t* y_off, int B,
                               int N, int D, int dt, void* y, float* y_inv, hipStream_t stream, const int32_t* pos,
                               int32_t* y_pos)
{
    const long rowbytes = (long)D * (dt == kBf16 ? 2 : 4);
    const int rpb = rows_per_block_for(rowbytes);
    dim3 grid((N + rpb - 1) / rpb, B);
    const uint8_t* xp = static_cast<const uint8_t*>(x);
    uint8_t* yp = static_cast<uint8_t*>(y);
    if (y_inv) {
        const int rows = kRowThreads / inv_lanes((int)(rowbytes / 16));
        const dim3 igrid((N + rows - 1) / rows, B);
        if (dt == kBf16)
            hipLaunchKernelGGL(pair_average_inv_kernel<Bf16>, igrid, dim3(kRowThreads), 0, stream, xp, x_off, src,
                               y_off, N, D, yp, y_inv, pos, y_pos);
        else
            hipLaunchKernelGGL(pair_average_inv_kernel<F32>, igrid, dim3(kRowThreads), 0, stream, xp, x_off, src,
                               y_off, N, D, yp, y_inv, pos, y_pos);
        return hipGetLastError();
    }
    if (dt == kBf16)
        hipLaunchKernelGGL(pair_average_kernel<Bf16>, grid, dim3(kRowThreads), 0, stream, xp, x_off, src, y_off, N, D,
                           rpb, yp, pos, y_pos);
    else
        hipLaunchKernelGGL(pair_average_kernel<F32>, grid, dim3(kRowThreads), 0, stream, xp, x_off, src, y_off, N, D,
                           rpb, yp, pos, y_pos);
    return hipGetLastError();
}

hipError_t launch_compose(const int32_t* map_a, const int32_t* map_b, int B, int N, int32_t* map_ab,
                          hipStream_t stream)
{
    const long total = (long)B * N;
    dim3 grid((unsigned)((total + kRowThreads - 1) / kRowThreads));
    hipLaunchKernelGGL(compose_kernel, grid, dim3(kRowThreads), 0, stream, map_a, map_b, N, total, map_ab);
    return hipGetLastError();
}

hipError_t launch_unmerge(const void* z, const int32_t* z_off, const int32_t* map, const void* z_spec, int E, int B,
                          int N, int D, int dt, void* out, hipStream_t stream, const int32_t* map2, int32_t* map_ab)
{
    const long rowbytes = (long)D * (dt == kBf16 ? 2 : 4);
    const int rpb = rows_per_block_for(rowbytes, kGatherBytesPerBlock);
    const int nx = (E + N + rpb - 1) / rpb;
    // XCD-major where a batch covers every XCD and an image's rows fit in one XCD's L2.
    const bool xcd_major = B >= kXcdCount && (long)N * rowbytes <= kXcdL2Bytes;
    const dim3 grid = xcd_major ? dim3((unsigned)((long)nx * ((B + kXcdCount - 1) / kXcdCount) * kXcdCount), 1)
                                : dim3((unsigned)nx, (unsigned)B);
    const uint8_t* zp = static_cast<const uint8_t*>(z);
    const uint8_t* sp = static_cast<const uint8_t*>(z_spec);
    uint8_t* op = static_cast<uint8_t*>(out);
    if (dt == kBf16)
        hipLaunchKernelGGL(unmerge_kernel<Bf16>, grid, dim3(kRowThreads), 0, stream, zp, z_off, map, map2, map_ab, sp, E,
                           N, D, rpb, op, B, xcd_major ? 1 : 0);
    else
        hipLaunchKernelGGL(unmerge_kernel<F32>, grid, dim3(kRowThreads), 0, stream, zp, z_off, map, map2, map_ab, sp, E,
                           N, D, rpb, op, B, xcd_major ? 1 : 0);
    return hipGetLastError();
}

}  // namespace mpm

namespace mpm {

hipError_t launch_pad(const void* z, const int32_t* z_off, int B, int P, long rowbytes, void* out, bool unpad,
                      hipStream_t stream)
{
    const int rpb = rows_per_block_for(rowbytes, kGatherBytesPerBlock);
    dim3 grid((P + rpb - 1) / rpb, B);
    const uint8_t* zp = static_cast<const uint8_t*>(z);
    uint8_t* op = static_cast<uint8_t*>(out);
    if (unpad)
        hipLaunchKernelGGL(pad_kernel<true>, grid, dim3(kRowThreads), 0, stream, zp, z_off, P, rowbytes, rpb, op);
    else
        hipLaunchKernelGGL(pad_kernel<false>, grid, dim3(kRowThreads), 0, stream, zp, z_off, P, rowbytes, rpb, op);
    return hipGetLastError();
}

}  // namespace mpm
