// Fused cosine affinity + self-masked row argmax (Eq. 1 and the nearest
// neighbour of Sec. 3.2) for gfx950.
//
// For image b with n tokens, every query i gets
//     nb[i] = argmax_{j != i, j < n} (x_i . x_j) * inv_j,   inv_j = 1 / max(||x_j||, 1e-12),
// with the lowest j kept among equal scores. Dividing the dot product by
// ||x_i|| as well would not move a row's argmax, so only the candidate norm is
// applied. The dot products come from MFMA on the stored values (bfloat16
// products are exact in float32, accumulation is float32); normalising first
// and rounding the unit vectors back to bfloat16 would cost about three
// decimal digits of the cosine, so the inputs are never rescaled.
//
// Tiling. A workgroup owns QT queries of one image and streams every
// candidate tile of CT tokens past them; the N x N affinity only ever lives
// in MFMA accumulators. Per candidate tile the K dimension (D) is staged
// through LDS in 128-byte chunks, double-buffered: the global loads of the
// next chunk are in flight while the current one feeds the MFMAs.
// In the 32x32 MFMA the candidate is the row operand and the query the column
// operand, so each lane's 16 accumulator values belong to ONE query and 16
// different candidates: the running (max, index) reduction is per lane, in
// registers, in ascending candidate order, and lanes/waves are merged
// lexicographically (larger score, then smaller index) only once at the end.
// The candidate norms are accumulated from the same register fragments that
// feed the MFMAs (one wave row per candidate slice), so X is read once per
// tile and no separate normalisation pass exists.
#include "mpm_device.h"
#include "mpm_launch.h"

namespace mpm {
namespace {

template <class S>
struct Mfma;

template <>
struct Mfma<Bf16> {
    // 16 bytes per lane = 8 bfloat16 values along k: one 32x32x16 MFMA.
    static __device__ __forceinline__ void mma(f32x16& acc, u32x4 a, u32x4 b)
    {
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
    }
    static __device__ __forceinline__ float sumsq(u32x4 a, float s)
    {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float lo = bf16_lo(a[e]);
            const float hi = bf16_hi(a[e]);
            s = fmaf(lo, lo, s);
            s = fmaf(hi, hi, s);
        }
        return s;
    }
};

template <>
struct Mfma<F32> {
    // 16 bytes per lane = 4 float32 values along k: four 32x32x2 MFMAs. Lane l
    // feeds k-slot l/32 of the instruction; both operands use the same
    // lane -> k assignment, so the sum runs over all 8 k of the 32-byte group.
    static __device__ __forceinline__ void mma(f32x16& acc, u32x4 a, u32x4 b)
    {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[e]), __uint_as_float(b[e]),
                                                       acc, 0, 0, 0);
    }
    static __device__ __forceinline__ float sumsq(u32x4 a, float s)
    {
#pragma unroll
        for (int e = 0; e < 4; ++e) s = fmaf(__uint_as_float(a[e]), __uint_as_float(a[e]), s);
        return s;
    }
};

constexpr int kXcds = 8;  // MI355X: workgroups are dealt round-robin to 8 XCDs, each with its own L2

// WC x WQ waves; each wave computes MT x NT tiles of 32 candidates x 32 queries;
// CHUNK bytes of the K dimension are staged per LDS buffer.
template <class S, int WC, int WQ, int MT, int NT, int CHUNK>
__global__ __launch_bounds__(WC * WQ * kWave) void affinity_argmax_kernel(
    const uint8_t* __restrict__ x, const int32_t* __restrict__ x_off, int B, int N, int D, int qblocks,
    int xcd_major, int32_t* __restrict__ nb, float* __restrict__ best)
{
    constexpr int THREADS = WC * WQ * kWave;
    constexpr int CT = WC * MT * 32;     // candidates per tile
    constexpr int QT = WQ * NT * 32;     // queries per workgroup
    constexpr int STRIDE = CHUNK + 16;   // padded LDS row pitch (bytes)
    constexpr int VPR = CHUNK / 16;      // 16-byte vectors per row per stage
    constexpr int CLOADS = CT * VPR / THREADS;
    constexpr int QLOADS = QT * VPR / THREADS;
    static_assert(CT * VPR % THREADS == 0 && QT * VPR % THREADS == 0, "tile/thread mismatch");

    __shared__ __attribute__((aligned(16))) uint8_t lds_c[2][CT * STRIDE];
    __shared__ __attribute__((aligned(16))) uint8_t lds_q[2][QT * STRIDE];
    __shared__ __attribute__((aligned(16))) float inv_c[2][CT];
    __shared__ float red_v[WC][QT];
    __shared__ int32_t red_i[WC][QT];

    // Workgroup -> (image, query block). With xcd_major, consecutive ids that the
    // hardware sends to the same XCD walk through the query blocks of one image
    // before the next, so an image's candidate tiles are re-read from that XCD's L2.
    int b, qb;
    if (xcd_major) {
        const int xcd = blockIdx.x % kXcds;
        const int slot = blockIdx.x / kXcds;
        b = xcd + kXcds * (slot / qblocks);
        qb = slot % qblocks;
    } else {
        b = blockIdx.x / qblocks;
        qb = blockIdx.x % qblocks;
    }
    if (b >= B) return;
    const int qbase = qb * QT;
    const int row0 = x_off ? x_off[b] : b * N;
    const int n = x_off ? x_off[b + 1] - row0 : N;
    if (qbase >= n) return;  // uniform over the workgroup, before any barrier

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wc = wave % WC;
    const int wq = wave / WC;
    const int lrow = lane & 31;   // operand row inside a 32-row MFMA tile
    const int khalf = lane >> 5;  // which 16-byte half of a 32-byte k group

    const long rowbytes = (long)D * S::kBytes;
    const uint8_t* ximg = x + (long)row0 * rowbytes;
    const int nchunks = (int)((rowbytes + CHUNK - 1) / CHUNK);
    const int ntiles = (n + CT - 1) / CT;
    const int total = ntiles * nchunks;

    u32x4 pc[CLOADS];
    u32x4 pq[QLOADS];
    const u32x4 zero = {0u, 0u, 0u, 0u};

    auto gload = [&](int step) {
        const int tile = step / nchunks;
        const long kb = (long)(step - tile * nchunks) * CHUNK;
#pragma unroll
        for (int u = 0; u < CLOADS; ++u) {
            const int slot = tid + u * THREADS;
            const int r = slot / VPR;
            const long kk = kb + (slot % VPR) * 16;
            const int row = tile * CT + r;
            pc[u] = (row < n && kk < rowbytes) ? load16(ximg + row * rowbytes + kk) : zero;
        }
#pragma unroll
        for (int u = 0; u < QLOADS; ++u) {
            const int slot = tid + u * THREADS;
            const int r = slot / VPR;
            const long kk = kb + (slot % VPR) * 16;
            const int row = qbase + r;
            pq[u] = (row < n && kk < rowbytes) ? load16(ximg + row * rowbytes + kk) : zero;
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int u = 0; u < CLOADS; ++u) {
            const int slot = tid + u * THREADS;
            store16(&lds_c[buf][(slot / VPR) * STRIDE + (slot % VPR) * 16], pc[u]);
        }
#pragma unroll
        for (int u = 0; u < QLOADS; ++u) {
            const int slot = tid + u * THREADS;
            store16(&lds_q[buf][(slot / VPR) * STRIDE + (slot % VPR) * 16], pq[u]);
        }
    };

    f32x16 acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x16{};
    float ss[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) ss[mt] = 0.0f;
    float bv[NT];
    int32_t bi[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        bv[nt] = -__builtin_inff();
        bi[nt] = -1;
    }

    gload(0);
    lstore(0);
    __syncthreads();

    for (int step = 0; step < total; ++step) {
        const int buf = step & 1;
        if (step + 1 < total) gload(step + 1);

        const uint8_t* lc = lds_c[buf] + (wc * MT * 32 + lrow) * STRIDE + khalf * 16;
        const uint8_t* lq = lds_q[buf] + (wq * NT * 32 + lrow) * STRIDE + khalf * 16;
#pragma unroll
        for (int g = 0; g < CHUNK / 32; ++g) {
            u32x4 a[MT], q[NT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                a[mt] = *reinterpret_cast<const u32x4*>(lc + mt * 32 * STRIDE + g * 32);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                q[nt] = *reinterpret_cast<const u32x4*>(lq + nt * 32 * STRIDE + g * 32);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) Mfma<S>::mma(acc[mt][nt], a[mt], q[nt]);
            // Candidate norms: m-tile mt is summed by the wave with wq == mt % WQ only.
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                if (mt % WQ == wq) ss[mt] = Mfma<S>::sumsq(a[mt], ss[mt]);
        }

        const int tile = step / nchunks;
        const bool tile_end = (step - tile * nchunks) == nchunks - 1;
        if (tile_end) {
            // Lanes l and l+32 hold the two k halves of candidate row lrow.
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                if (mt % WQ != wq) continue;
                const float t = ss[mt] + __shfl_xor(ss[mt], 32);
                ss[mt] = 0.0f;
                if (khalf == 0) inv_c[tile & 1][wc * MT * 32 + mt * 32 + lrow] = 1.0f / fmaxf(sqrtf(t), 1e-12f);
            }
        }
        if (step + 1 < total) lstore(buf ^ 1);
        __syncthreads();

        if (tile_end) {
            // Epilogue: scale by the candidate's inverse norm, mask, running argmax.
            const int cb = tile * CT;
            const float* iv = inv_c[tile & 1];
            const bool need_mask = (cb + CT > n) || (cb < qbase + QT && qbase < cb + CT);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int qi = qbase + wq * NT * 32 + nt * 32 + lrow;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        // Accumulator element 4g+e of this lane is candidate row 8g + 4*khalf + e.
                        const int jl = wc * MT * 32 + mt * 32 + 8 * g + 4 * khalf;
                        const f32x4 ivv = *reinterpret_cast<const f32x4*>(&iv[jl]);
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float s = acc[mt][nt][4 * g + e] * ivv[e];
                            const int j = cb + jl + e;
                            const bool ok = !need_mask || (j < n && j != qi);
                            if (ok && s > bv[nt]) {
                                bv[nt] = s;
                                bi[nt] = j;
                            }
                        }
                    }
                    acc[mt][nt] = f32x16{};
                }
            }
        }
    }

    // Merge the two lane halves (same query, interleaved candidate rows), then
    // the WC candidate waves, lexicographically: larger score, then smaller index.
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        float v = bv[nt];
        int32_t i = bi[nt];
        const float ov = __shfl_xor(v, 32);
        const int32_t oi = __shfl_xor(i, 32);
        if (ov > v || (ov == v && (uint32_t)oi < (uint32_t)i)) {
            v = ov;
            i = oi;
        }
        if (khalf == 0) {
            const int ql = wq * NT * 32 + nt * 32 + lrow;
            red_v[wc][ql] = v;
            red_i[wc][ql] = i;
        }
    }
    __syncthreads();
    for (int ql = tid; ql < QT; ql += THREADS) {
        const int qi = qbase + ql;
        if (qi >= n) continue;
        float v = red_v[0][ql];
        int32_t i = red_i[0][ql];
#pragma unroll
        for (int w = 1; w < WC; ++w) {
            const float ov = red_v[w][ql];
            const int32_t oi = red_i[w][ql];
            if (ov > v || (ov == v && (uint32_t)oi < (uint32_t)i)) {
                v = ov;
                i = oi;
            }
        }
        nb[(long)b * N + qi] = i;
        if (best) {
            // Diagnostic only: divide by the query's own norm to report the cosine.
            const uint8_t* xr = ximg + qi * rowbytes;
            float t = 0.0f;
            for (long kk = 0; kk < rowbytes; kk += 16) t = Mfma<S>::sumsq(load16(xr + kk), t);
            best[(long)b * N + qi] = i >= 0 ? v / fmaxf(sqrtf(t), 1e-12f) : -__builtin_inff();
        }
    }
}

template <class S, int WC, int WQ, int MT, int NT, int CHUNK>
hipError_t launch_t(const void* x, const int32_t* x_off, int B, int N, int D, int32_t* nb, float* best,
                    hipStream_t stream)
{
    constexpr int QT = WQ * NT * 32;
    const int qblocks = (N + QT - 1) / QT;
    const int xcd_major = B >= kXcds ? 1 : 0;
    const long groups = xcd_major ? (long)kXcds * ((B + kXcds - 1) / kXcds) * qblocks : (long)B * qblocks;
    hipLaunchKernelGGL((affinity_argmax_kernel<S, WC, WQ, MT, NT, CHUNK>), dim3((unsigned)groups),
                       dim3(WC * WQ * kWave), 0, stream, static_cast<const uint8_t*>(x), x_off, B, N, D, qblocks,
                       xcd_major, nb, best);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_argmax(const void* x, const int32_t* x_off, int B, int N, int D, int dt, int32_t* nb,
                         float* best, hipStream_t stream)
{
    if (dt == kBf16) return launch_t<Bf16, 2, 4, 4, 2, 128>(x, x_off, B, N, D, nb, best, stream);
    return launch_t<F32, 2, 2, 2, 2, 128>(x, x_off, B, N, D, nb, best, stream);
}

}  // namespace mpm
