// Generic 3D convolution as an implicit GEMM on MFMA, any kernel size,
// stride and padding, float32 or bfloat16 storage.
//
// forward:  rows = output voxels (n, o), cols = C_out, K = C_in * k^3
//           A[m][(ci,t)] = x[n, ci, o*s - p + t]   (gathered, zero outside)
//           B[(ci,t)][co] = w[co, ci, t]           (contiguous in K)
// dgrad:    rows = input voxels (n, i), cols = C_in, K = C_out * k^3
//           A[m][(co,t)] = dy[n, co, (i + p - t)/s] when divisible and in range
//           B[(co,t)][ci] = w[co, ci, t]
// wgrad:    rows = C_out, cols = C_in * k^3, K = output voxels (split over
//           workgroups; partial tiles reduced in a fixed order afterwards)
//           A[co][(n,o)] = dy[n, co, o],  B[(n,o)][(ci,t)] = x[n, ci, o*s - p + t]
//
// Workgroup tile 64 x 64, four waves of 32 x 32 (2 x 2 MFMA 16x16 tiles).
// Each K step stages a 64 x BK slab of A and of B in LDS with the K index
// innermost, so that every lane fetches its MFMA operand with one 16-byte
// LDS read: bf16 uses v_mfma_f32_16x16x32_bf16 (8 K values per lane),
// float32 uses four v_mfma_f32_16x16x4_f32 (4 K values per lane).
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "vec.hpp"
#include "prof.hpp"

namespace rat3d {

template <typename T> struct MfmaCfg;
template <> struct MfmaCfg<bf16> { static constexpr int KV = 8, BK = 32; };
template <> struct MfmaCfg<float> { static constexpr int KV = 4, BK = 16; };

union Frag16 {
    uint4 u;
    bf16x8 b;
    float f[4];
    bf16 h[8];
};

template <typename T> __device__ __forceinline__ void mma16(f32x4& acc, const Frag16& a,
                                                            const Frag16& b);
template <> __device__ __forceinline__ void mma16<bf16>(f32x4& acc, const Frag16& a,
                                                        const Frag16& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.b, b.b, acc, 0, 0, 0);
}
template <> __device__ __forceinline__ void mma16<float>(f32x4& acc, const Frag16& a,
                                                         const Frag16& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.f[0], b.f[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.f[1], b.f[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.f[2], b.f[2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.f[3], b.f[3], acc, 0, 0, 0);
}

constexpr int kRow = 80;  // LDS bytes per staged row: 64 bytes of K values + 16 pad

template <typename T>
__device__ __forceinline__ void store_frag(unsigned char* lds, const T (&v)[16 / sizeof(T)]) {
    Frag16 f;
#pragma unroll
    for (int j = 0; j < (int)(16 / sizeof(T)); ++j) {
        if constexpr (sizeof(T) == 2) f.h[j] = (bf16)v[j];
        else f.f[j] = (float)v[j];
    }
    *reinterpret_cast<uint4*>(lds) = f.u;
}

// One K step of the 64x64 tile: each wave multiplies its 32x32 quarter.
template <typename T>
__device__ __forceinline__ void tile_mma(const unsigned char* As, const unsigned char* Bs,
                                         f32x4 (&acc)[2][2], int lane, int wm, int wn) {
    Frag16 a[2], b[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        a[i].u = *reinterpret_cast<const uint4*>(As + (wm * 32 + i * 16 + (lane & 15)) * kRow +
                                                 (lane >> 4) * 16);
        b[i].u = *reinterpret_cast<const uint4*>(Bs + (wn * 32 + i * 16 + (lane & 15)) * kRow +
                                                 (lane >> 4) * 16);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) mma16<T>(acc[i][j], a[i], b[j]);
}

// ---------------------------------------------------------------- fwd / dgrad
template <typename T, bool DGRAD>
__global__ __launch_bounds__(256) void conv_gather_fd(ConvGeom g, const T* __restrict__ src,
                                                      const T* __restrict__ wt,
                                                      const float* __restrict__ bias,
                                                      T* __restrict__ dst, int accumulate) {
    constexpr int KV = MfmaCfg<T>::KV, BK = MfmaCfg<T>::BK;
    __shared__ __align__(16) unsigned char As[64 * kRow];
    __shared__ __align__(16) unsigned char Bs[64 * kRow];
    __shared__ int4 ktab[BK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    // GEMM rows are voxels of the destination tensor.
    const int RD = DGRAD ? g.D : g.Do, RH = DGRAD ? g.H : g.Ho, RW = DGRAD ? g.W : g.Wo;
    const int64_t Vrow = (int64_t)RD * RH * RW;
    const int64_t M = (int64_t)g.N * Vrow;
    const int Ncol = DGRAD ? g.Ci : g.Co;
    const int Csrc = DGRAD ? g.Co : g.Ci;
    const int SD = DGRAD ? g.Do : g.D, SH = DGRAD ? g.Ho : g.H, SW = DGRAD ? g.Wo : g.W;
    const int64_t Vsrc = (int64_t)SD * SH * SW;
    const int KT = g.k * g.k * g.k;
    const int K = Csrc * KT;
    const int64_t m0 = (int64_t)blockIdx.x * 64;
    const int c0 = blockIdx.y * 64;

    const int ar = tid >> 2, aq = tid & 3;
    const int64_t am = m0 + ar;
    const bool arow_ok = am < M;
    int a_d = 0, a_h = 0, a_w = 0;
    int64_t a_base = 0;
    if (arow_ok) {
        const int64_t n = am / Vrow;
        int64_t sp = am - n * Vrow;
        a_d = (int)(sp / ((int64_t)RH * RW));
        sp -= (int64_t)a_d * RH * RW;
        a_h = (int)(sp / RW);
        a_w = (int)(sp - (int64_t)a_h * RW);
        a_base = n * Csrc * Vsrc;
    }
    const int bcol = c0 + (tid >> 2), bq = tid & 3;

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = 0; k0 < K; k0 += BK) {
        if (tid < BK) {
            const int k = k0 + tid;
            int4 e = make_int4(-1, 0, 0, 0);
            if (k < K) {
                const int c = k / KT;
                const int t = k - c * KT;
                const int kd = t / (g.k * g.k);
                const int r = t - kd * g.k * g.k;
                const int kh = r / g.k;
                e = make_int4(c, kd, kh, r - kh * g.k);
            }
            ktab[tid] = e;
        }
        __syncthreads();
        {
            T v[KV];
#pragma unroll
            for (int j = 0; j < KV; ++j) {
                const int4 e = ktab[aq * KV + j];
                T val = Elt<T>::to_bits(0.f);
                if (arow_ok && e.x >= 0) {
                    if constexpr (!DGRAD) {
                        const int id = a_d * g.s - g.p + e.y, ih = a_h * g.s - g.p + e.z,
                                  iw = a_w * g.s - g.p + e.w;
                        if ((unsigned)id < (unsigned)g.D && (unsigned)ih < (unsigned)g.H &&
                            (unsigned)iw < (unsigned)g.W)
                            val = src[a_base + e.x * Vsrc + ((int64_t)id * g.H + ih) * g.W + iw];
                    } else {
                        const int nd = a_d + g.p - e.y, nh = a_h + g.p - e.z,
                                  nw = a_w + g.p - e.w;
                        if (nd >= 0 && nh >= 0 && nw >= 0 && nd % g.s == 0 && nh % g.s == 0 &&
                            nw % g.s == 0) {
                            const int od = nd / g.s, oh = nh / g.s, ow = nw / g.s;
                            if (od < g.Do && oh < g.Ho && ow < g.Wo)
                                val = src[a_base + e.x * Vsrc + ((int64_t)od * g.Ho + oh) * g.Wo +
                                          ow];
                        }
                    }
                }
                v[j] = val;
            }
            store_frag<T>(As + ar * kRow + aq * 16, v);
        }
        {
            T v[KV];
#pragma unroll
            for (int j = 0; j < KV; ++j) {
                const int k = k0 + bq * KV + j;
                T val = Elt<T>::to_bits(0.f);
                if (bcol < Ncol && k < K) {
                    if constexpr (!DGRAD) {
                        val = wt[(int64_t)bcol * K + k];
                    } else {
                        const int co = ktab[bq * KV + j].x;
                        val = wt[((int64_t)co * g.Ci + bcol) * KT + (k - co * KT)];
                    }
                }
                v[j] = val;
            }
            store_frag<T>(Bs + (tid >> 2) * kRow + bq * 16, v);
        }
        __syncthreads();
        tile_mma<T>(As, Bs, acc, lane, wm, wn);
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = wm * 32 + i * 16 + 4 * (lane >> 4) + e;
                const int col = wn * 32 + j * 16 + (lane & 15);
                const int64_t m = m0 + row;
                const int c = c0 + col;
                if (m < M && c < Ncol) {
                    const int64_t n = m / Vrow, sp = m - n * Vrow;
                    const int64_t off = (n * Ncol + c) * Vrow + sp;
                    float v = acc[i][j][e];
                    if (bias) v += bias[c];
                    if (accumulate) v += Elt<T>::ld(dst + off);
                    Elt<T>::st(dst + off, v);
                }
            }
}

// Forward, bfloat16, source channels a multiple of 32 (every K step of 32
// is whole): the same 64 x 64 tiles, pipelined.  The next K step's operands
// are loaded into registers (unconditionally: taps outside the volume read
// element 0 and are zeroed) while the current step multiplies from one of
// two LDS buffers, so a step costs one barrier and no exposed load latency.
// A thread's 8 K values are consecutive taps of one or two channels: the
// channel and tap of the first come from one division, the rest by stepping
// the tap with a wrap; a tap's (kd, kh, kw) come from a table in LDS.
constexpr int kGatherMaxTaps = 343;
__global__ __launch_bounds__(256) void conv_gather_fwd_pipe(ConvGeom g, const bf16* __restrict__ src,
                                                            const bf16* __restrict__ wt,
                                                            const float* __restrict__ bias,
                                                            bf16* __restrict__ dst) {
    constexpr int KV = 8, BK = 32;
    __shared__ __align__(16) unsigned char As[2][64 * kRow];
    __shared__ __align__(16) unsigned char Bs[2][64 * kRow];
    __shared__ int taps[kGatherMaxTaps];  // kd | kh << 8 | kw << 16

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int KT = g.k * g.k * g.k, K = g.Ci * KT;
    const int64_t Vrow = (int64_t)g.Do * g.Ho * g.Wo, M = (int64_t)g.N * Vrow;
    const int64_t Vsrc = (int64_t)g.D * g.H * g.W;
    const int64_t m0 = (int64_t)blockIdx.x * 64;
    const int c0 = blockIdx.y * 64;
    for (int t = tid; t < KT; t += 256) {
        const int kd = t / (g.k * g.k), r = t - kd * g.k * g.k, kh = r / g.k;
        taps[t] = kd | kh << 8 | (r - kh * g.k) << 16;
    }

    // this thread's A row (an output voxel) and B row (an output channel)
    const int ar = tid >> 2, aq = tid & 3;
    const int64_t am = m0 + ar;
    const bool arow_ok = am < M;
    int id0 = 0, ih0 = 0, iw0 = 0;
    int64_t a_base = 0;
    {
        const int64_t mm = arow_ok ? am : 0;
        const int64_t n = mm / Vrow;
        int64_t sp = mm - n * Vrow;
        const int od = (int)(sp / ((int64_t)g.Ho * g.Wo));
        sp -= (int64_t)od * g.Ho * g.Wo;
        const int oh = (int)(sp / g.Wo), ow = (int)(sp - (int64_t)oh * g.Wo);
        id0 = od * g.s - g.p;
        ih0 = oh * g.s - g.p;
        iw0 = ow * g.s - g.p;
        a_base = n * g.Ci * Vsrc;
    }
    const int bcol = c0 + (tid >> 2);
    const bool bcol_ok = bcol < g.Co;
    const bf16* wrow = wt + (int64_t)(bcol_ok ? bcol : 0) * K;

    uint32_t av[KV / 2];
    uint4 bv;
    auto load = [&](int k0) {
        const int kf = k0 + aq * KV;
        int c = kf / KT, t = kf - c * KT;
        bf16 v[KV];
#pragma unroll
        for (int j = 0; j < KV; ++j) {
            const int e = taps[t];
            const int id = id0 + (e & 0xff), ih = ih0 + ((e >> 8) & 0xff), iw = iw0 + (e >> 16);
            const bool ok = arow_ok && (unsigned)id < (unsigned)g.D &&
                            (unsigned)ih < (unsigned)g.H && (unsigned)iw < (unsigned)g.W;
            const int64_t off = ok ? a_base + c * Vsrc + ((int64_t)id * g.H + ih) * g.W + iw : 0;
            const bf16 x = src[off];
            v[j] = ok ? x : (bf16)0;
            if (++t == KT) {
                t = 0;
                ++c;
            }
        }
#pragma unroll
        for (int j = 0; j < KV / 2; ++j) av[j] = (uint32_t)v[2 * j] | (uint32_t)v[2 * j + 1] << 16;
        const uint4 w4 = *reinterpret_cast<const uint4*>(wrow + k0 + aq * KV);
        bv = bcol_ok ? w4 : make_uint4(0u, 0u, 0u, 0u);
    };
    auto stage = [&](int buf) {
        *reinterpret_cast<uint4*>(As[buf] + ar * kRow + aq * 16) = make_uint4(av[0], av[1], av[2], av[3]);
        *reinterpret_cast<uint4*>(Bs[buf] + (tid >> 2) * kRow + aq * 16) = bv;
    };

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    __syncthreads();  // the tap table
    const int S = K / BK;
    load(0);
    stage(0);
    __syncthreads();
    for (int st = 0; st < S; ++st) {
        const bool more = st + 1 < S;
        if (more) load((st + 1) * BK);
        tile_mma<bf16>(As[st & 1], Bs[st & 1], acc, lane, wm, wn);
        if (more) stage((st + 1) & 1);
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = wm * 32 + i * 16 + 4 * (lane >> 4) + e;
                const int col = wn * 32 + j * 16 + (lane & 15);
                const int64_t m = m0 + row;
                const int c = c0 + col;
                if (m < M && c < g.Co) {
                    const int64_t n = m / Vrow, sp = m - n * Vrow;
                    float v = acc[i][j][e];
                    if (bias) v += bias[c];
                    dst[(n * g.Co + c) * Vrow + sp] = f2bf(v);
                }
            }
}

// ---------------------------------------------------------------- strided dgrad
// Input gradient of a strided convolution, decomposed by phase: input voxel
// i (per axis) receives from tap t only when s divides i + p - t, i.e. when
// t = (i + p) mod s (mod s).  The voxels of one residue class r = i mod s per
// axis therefore share one tap set (t0 + s j < k, t0 = (r + p) mod s), and
// for such a voxel i = r + s m the source position is od = m + (r + p - t)/s.
// blockIdx.z picks the class (rd, rh, rw); its rows are the class's voxels
// (n, md, mh, mw) and its K the Co x (its taps) products, so no product is a
// structural zero (the k^3 taps are split over the s^3 classes).  A class
// without taps (k < s) stores zeros (or leaves an accumulated dx unchanged).
template <typename T>
__global__ __launch_bounds__(256) void conv_gather_dgrad_phase(ConvGeom g,
                                                               const T* __restrict__ dy,
                                                               const T* __restrict__ wt,
                                                               T* __restrict__ dx,
                                                               int accumulate) {
    constexpr int KV = MfmaCfg<T>::KV, BK = MfmaCfg<T>::BK;
    __shared__ __align__(16) unsigned char As[64 * kRow];
    __shared__ __align__(16) unsigned char Bs[64 * kRow];
    __shared__ int4 ktab[BK];  // (co or -1, od offset, oh offset, ow offset)
    __shared__ int ttab[BK];   // flattened tap kd * k^2 + kh * k + kw

    const int s = g.s;
    const int cls = blockIdx.z;
    const int rd = cls / (s * s), rh = (cls / s) % s, rw = cls % s;
    // rows: the class's voxels; taps per axis
    const int Md = rd < g.D ? (g.D - rd + s - 1) / s : 0;
    const int Mh = rh < g.H ? (g.H - rh + s - 1) / s : 0;
    const int Mw = rw < g.W ? (g.W - rw + s - 1) / s : 0;
    const int t0d = (rd + g.p) % s, t0h = (rh + g.p) % s, t0w = (rw + g.p) % s;
    const int nd = t0d < g.k ? (g.k - t0d + s - 1) / s : 0;
    const int nh = t0h < g.k ? (g.k - t0h + s - 1) / s : 0;
    const int nw = t0w < g.k ? (g.k - t0w + s - 1) / s : 0;
    const int KTc = nd * nh * nw;
    const int Kc = g.Co * KTc;
    const int64_t Vc = (int64_t)Md * Mh * Mw;
    const int64_t M = (int64_t)g.N * Vc;
    const int64_t m0 = (int64_t)blockIdx.x * 64;
    if (m0 >= M) return;  // this class has fewer rows than the grid covers
    const int c0 = blockIdx.y * 64;
    const int KT = g.k * g.k * g.k;
    const int64_t Vsrc = (int64_t)g.Do * g.Ho * g.Wo;
    const int64_t Vdst = (int64_t)g.D * g.H * g.W;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int ar = tid >> 2, aq = tid & 3;
    const int64_t am = m0 + ar;
    const bool arow_ok = am < M;
    int a_d = 0, a_h = 0, a_w = 0;
    int64_t a_base = 0;
    if (arow_ok) {
        const int64_t n = am / Vc;
        int64_t sp = am - n * Vc;
        a_d = (int)(sp / ((int64_t)Mh * Mw));
        sp -= (int64_t)a_d * Mh * Mw;
        a_h = (int)(sp / Mw);
        a_w = (int)(sp - (int64_t)a_h * Mw);
        a_base = n * g.Co * Vsrc;
    }
    const int bcol = c0 + (tid >> 2), bq = tid & 3;

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = 0; k0 < Kc; k0 += BK) {
        if (tid < BK) {
            const int k = k0 + tid;
            int4 e = make_int4(-1, 0, 0, 0);
            int t = 0;
            if (k < Kc) {
                const int co = k / KTc;
                int r = k - co * KTc;
                const int jd = r / (nh * nw);
                r -= jd * nh * nw;
                const int jh = r / nw, jw = r - (r / nw) * nw;
                const int td = t0d + s * jd, th = t0h + s * jh, tw = t0w + s * jw;
                e = make_int4(co, (rd + g.p - td) / s, (rh + g.p - th) / s, (rw + g.p - tw) / s);
                t = (td * g.k + th) * g.k + tw;
            }
            ktab[tid] = e;
            ttab[tid] = t;
        }
        __syncthreads();
        {
            T v[KV];
#pragma unroll
            for (int j = 0; j < KV; ++j) {
                const int4 e = ktab[aq * KV + j];
                T val = Elt<T>::to_bits(0.f);
                if (arow_ok && e.x >= 0) {
                    const int od = a_d + e.y, oh = a_h + e.z, ow = a_w + e.w;
                    if ((unsigned)od < (unsigned)g.Do && (unsigned)oh < (unsigned)g.Ho &&
                        (unsigned)ow < (unsigned)g.Wo)
                        val = dy[a_base + e.x * Vsrc + ((int64_t)od * g.Ho + oh) * g.Wo + ow];
                }
                v[j] = val;
            }
            store_frag<T>(As + ar * kRow + aq * 16, v);
        }
        {
            T v[KV];
#pragma unroll
            for (int j = 0; j < KV; ++j) {
                const int kk = bq * KV + j;
                T val = Elt<T>::to_bits(0.f);
                const int co = ktab[kk].x;
                if (bcol < g.Ci && co >= 0)
                    val = wt[((int64_t)co * g.Ci + bcol) * KT + ttab[kk]];
                v[j] = val;
            }
            store_frag<T>(Bs + (tid >> 2) * kRow + bq * 16, v);
        }
        __syncthreads();
        tile_mma<T>(As, Bs, acc, lane, wm, wn);
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = wm * 32 + i * 16 + 4 * (lane >> 4) + e;
                const int col = wn * 32 + j * 16 + (lane & 15);
                const int64_t m = m0 + row;
                const int c = c0 + col;
                if (m < M && c < g.Ci) {
                    const int64_t n = m / Vc;
                    int64_t sp = m - n * Vc;
                    const int md = (int)(sp / ((int64_t)Mh * Mw));
                    sp -= (int64_t)md * Mh * Mw;
                    const int mh = (int)(sp / Mw), mw = (int)(sp - (sp / Mw) * Mw);
                    const int64_t off = (n * g.Ci + c) * Vdst +
                                        ((int64_t)(rd + s * md) * g.H + rh + s * mh) * g.W + rw +
                                        s * mw;
                    float v = acc[i][j][e];
                    if (accumulate) v += Elt<T>::ld(dx + off);
                    Elt<T>::st(dx + off, v);
                }
            }
}

// The strided input gradient in bf16 with C_out (the channels its K runs
// over) a multiple of 32, pipelined like conv_gather_fwd_pipe: the
// class's taps (at most (k / s + 1)^3) in an LDS table built once, each
// thread's 8 consecutive K values (co, tap) stepped through it, the next K
// step's loads issued unconditionally before the current step's MFMAs into
// the other of two LDS buffers.
constexpr int kPhaseMaxTaps = 64;
__global__ __launch_bounds__(256) void conv_gather_dgrad_phase_pipe(ConvGeom g,
                                                                    const bf16* __restrict__ dy,
                                                                    const bf16* __restrict__ wt,
                                                                    bf16* __restrict__ dx,
                                                                    int accumulate) {
    constexpr int KV = 8, BK = 32;
    __shared__ __align__(16) unsigned char As[2][64 * kRow];
    __shared__ __align__(16) unsigned char Bs[2][64 * kRow];
    __shared__ int toff[kPhaseMaxTaps];  // od | oh << 8 | ow << 16 offsets (each + 128)
    __shared__ int tflat[kPhaseMaxTaps]; // flattened tap kd * k^2 + kh * k + kw

    const int s = g.s;
    const int cls = blockIdx.z;
    const int rd = cls / (s * s), rh = (cls / s) % s, rw = cls % s;
    const int Md = rd < g.D ? (g.D - rd + s - 1) / s : 0;
    const int Mh = rh < g.H ? (g.H - rh + s - 1) / s : 0;
    const int Mw = rw < g.W ? (g.W - rw + s - 1) / s : 0;
    const int t0d = (rd + g.p) % s, t0h = (rh + g.p) % s, t0w = (rw + g.p) % s;
    const int nd = t0d < g.k ? (g.k - t0d + s - 1) / s : 0;
    const int nh = t0h < g.k ? (g.k - t0h + s - 1) / s : 0;
    const int nw = t0w < g.k ? (g.k - t0w + s - 1) / s : 0;
    const int KTc = nd * nh * nw;
    const int Kc = g.Co * KTc;
    const int64_t Vc = (int64_t)Md * Mh * Mw;
    const int64_t M = (int64_t)g.N * Vc;
    const int64_t m0 = (int64_t)blockIdx.x * 64;
    if (m0 >= M) return;  // this class has fewer rows than the grid covers
    const int c0 = blockIdx.y * 64;
    const int KT = g.k * g.k * g.k;
    const int64_t Vsrc = (int64_t)g.Do * g.Ho * g.Wo;
    const int64_t Vdst = (int64_t)g.D * g.H * g.W;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    for (int j = tid; j < KTc; j += 256) {
        const int jd = j / (nh * nw), r = j - jd * nh * nw, jh = r / nw, jw = r - jh * nw;
        const int td = t0d + s * jd, th = t0h + s * jh, tw = t0w + s * jw;
        toff[j] = ((rd + g.p - td) / s + 128) | ((rh + g.p - th) / s + 128) << 8 |
                  ((rw + g.p - tw) / s + 128) << 16;
        tflat[j] = (td * g.k + th) * g.k + tw;
    }
    const int ar = tid >> 2, aq = tid & 3;
    const int64_t am = m0 + ar;
    const bool arow_ok = am < M;
    int a_d = 0, a_h = 0, a_w = 0;
    int64_t a_base = 0;
    if (arow_ok) {
        const int64_t n = am / Vc;
        int64_t sp = am - n * Vc;
        a_d = (int)(sp / ((int64_t)Mh * Mw));
        sp -= (int64_t)a_d * Mh * Mw;
        a_h = (int)(sp / Mw);
        a_w = (int)(sp - (int64_t)a_h * Mw);
        a_base = n * g.Co * Vsrc;
    }
    const int bcol = c0 + (tid >> 2);
    const bool bcol_ok = bcol < g.Ci;
    const int bc = bcol_ok ? bcol : 0;

    uint32_t av[KV / 2], bv[KV / 2];
    auto load = [&](int k0) {
        const int kf = k0 + aq * KV;
        int co = kf / KTc, j = kf - co * KTc;
        bf16 a[KV], b[KV];
#pragma unroll
        for (int q = 0; q < KV; ++q) {
            const int e = toff[j];
            const int od = a_d + (e & 0xff) - 128, oh = a_h + ((e >> 8) & 0xff) - 128,
                      ow = a_w + (e >> 16) - 128;
            const bool ok = arow_ok && (unsigned)od < (unsigned)g.Do &&
                            (unsigned)oh < (unsigned)g.Ho && (unsigned)ow < (unsigned)g.Wo;
            const int64_t off = ok ? a_base + co * Vsrc + ((int64_t)od * g.Ho + oh) * g.Wo + ow : 0;
            const bf16 xa = dy[off];
            a[q] = ok ? xa : (bf16)0;
            const bf16 xb = wt[((int64_t)co * g.Ci + bc) * KT + tflat[j]];
            b[q] = bcol_ok ? xb : (bf16)0;
            if (++j == KTc) {
                j = 0;
                ++co;
            }
        }
#pragma unroll
        for (int q = 0; q < KV / 2; ++q) {
            av[q] = (uint32_t)a[2 * q] | (uint32_t)a[2 * q + 1] << 16;
            bv[q] = (uint32_t)b[2 * q] | (uint32_t)b[2 * q + 1] << 16;
        }
    };
    auto stage = [&](int buf) {
        *reinterpret_cast<uint4*>(As[buf] + ar * kRow + aq * 16) = make_uint4(av[0], av[1], av[2], av[3]);
        *reinterpret_cast<uint4*>(Bs[buf] + (tid >> 2) * kRow + aq * 16) = make_uint4(bv[0], bv[1], bv[2], bv[3]);
    };

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    __syncthreads();  // the tap tables
    const int S = Kc / BK;
    if (S > 0) {
        load(0);
        stage(0);
    }
    __syncthreads();
    for (int st = 0; st < S; ++st) {
        const bool more = st + 1 < S;
        if (more) load((st + 1) * BK);
        tile_mma<bf16>(As[st & 1], Bs[st & 1], acc, lane, wm, wn);
        if (more) stage((st + 1) & 1);
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = wm * 32 + i * 16 + 4 * (lane >> 4) + e;
                const int col = wn * 32 + j * 16 + (lane & 15);
                const int64_t m = m0 + row;
                const int c = c0 + col;
                if (m < M && c < g.Ci) {
                    const int64_t n = m / Vc;
                    int64_t sp = m - n * Vc;
                    const int md = (int)(sp / ((int64_t)Mh * Mw));
                    sp -= (int64_t)md * Mh * Mw;
                    const int mh = (int)(sp / Mw), mw = (int)(sp - (sp / Mw) * Mw);
                    const int64_t off = (n * g.Ci + c) * Vdst +
                                        ((int64_t)(rd + s * md) * g.H + rh + s * mh) * g.W + rw +
                                        s * mw;
                    float v = acc[i][j][e];
                    if (accumulate) v += bf2f(dx[off]);
                    dx[off] = f2bf(v);
                }
            }
}

// ---------------------------------------------------------------- wgrad
template <typename T>
__global__ __launch_bounds__(256) void conv_gather_wgrad(ConvGeom g, const T* __restrict__ x,
                                                         const T* __restrict__ dy,
                                                         float* __restrict__ part,
                                                         int64_t kchunk) {
    constexpr int KV = MfmaCfg<T>::KV, BK = MfmaCfg<T>::BK;
    __shared__ __align__(16) unsigned char As[64 * kRow];
    __shared__ __align__(16) unsigned char Bs[64 * kRow];
    __shared__ int4 vtab[BK];    // (n or -1, od*s-p, oh*s-p, ow*s-p)
    __shared__ int64_t vdy[BK];  // n*Co*Vo + o

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int KT = g.k * g.k * g.k;
    const int Ncols = g.Ci * KT;
    const int64_t Vo = (int64_t)g.Do * g.Ho * g.Wo, Vi = (int64_t)g.D * g.H * g.W;
    const int64_t Ktot = (int64_t)g.N * Vo;
    const int64_t kbeg = (int64_t)blockIdx.z * kchunk;
    const int64_t kend = kbeg + kchunk < Ktot ? kbeg + kchunk : Ktot;
    const int co0 = blockIdx.x * 64, col0 = blockIdx.y * 64;

    const int aco = co0 + (tid >> 2), aq = tid & 3;
    const int bcol = col0 + (tid >> 2), bq = tid & 3;
    int b_ci = 0, b_kd = 0, b_kh = 0, b_kw = 0;
    const bool bcol_ok = bcol < Ncols;
    if (bcol_ok) {
        b_ci = bcol / KT;
        const int t = bcol - b_ci * KT;
        b_kd = t / (g.k * g.k);
        const int r = t - b_kd * g.k * g.k;
        b_kh = r / g.k;
        b_kw = r - b_kh * g.k;
    }

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int64_t v0 = kbeg; v0 < kend; v0 += BK) {
        if (tid < BK) {
            const int64_t v = v0 + tid;
            int4 e = make_int4(-1, 0, 0, 0);
            int64_t off = 0;
            if (v < kend) {
                const int64_t n = v / Vo;
                int64_t o = v - n * Vo;
                const int od = (int)(o / ((int64_t)g.Ho * g.Wo));
                const int64_t r = o - (int64_t)od * g.Ho * g.Wo;
                const int oh = (int)(r / g.Wo), ow = (int)(r - (int64_t)oh * g.Wo);
                e = make_int4((int)n, od * g.s - g.p, oh * g.s - g.p, ow * g.s - g.p);
                off = n * g.Co * Vo + o;
            }
            vtab[tid] = e;
            vdy[tid] = off;
        }
        __syncthreads();
        {
            T v[KV];
#pragma unroll
            for (int j = 0; j < KV; ++j) {
                T val = Elt<T>::to_bits(0.f);
                if (aco < g.Co && vtab[aq * KV + j].x >= 0)
                    val = dy[vdy[aq * KV + j] + (int64_t)aco * Vo];
                v[j] = val;
            }
            store_frag<T>(As + (tid >> 2) * kRow + aq * 16, v);
        }
        {
            T v[KV];
#pragma unroll
            for (int j = 0; j < KV; ++j) {
                T val = Elt<T>::to_bits(0.f);
                const int4 e = vtab[bq * KV + j];
                if (bcol_ok && e.x >= 0) {
                    const int id = e.y + b_kd, ih = e.z + b_kh, iw = e.w + b_kw;
                    if ((unsigned)id < (unsigned)g.D && (unsigned)ih < (unsigned)g.H &&
                        (unsigned)iw < (unsigned)g.W)
                        val = x[((int64_t)e.x * g.Ci + b_ci) * Vi + ((int64_t)id * g.H + ih) * g.W +
                                iw];
                }
                v[j] = val;
            }
            store_frag<T>(Bs + (tid >> 2) * kRow + bq * 16, v);
        }
        __syncthreads();
        tile_mma<T>(As, Bs, acc, lane, wm, wn);
    }

    float* out = part + (int64_t)blockIdx.z * g.Co * Ncols;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int co = co0 + wm * 32 + i * 16 + 4 * (lane >> 4) + e;
                const int col = col0 + wn * 32 + j * 16 + (lane & 15);
                if (co < g.Co && col < Ncols) out[(int64_t)co * Ncols + col] = acc[i][j][e];
            }
}

// Sums `splits` partial weight-gradient slabs in split order into dw; four
// consecutive elements per thread (count is a multiple of 4 on that path).
// dw (+)= sum of the split partials, float4 lanes.  A block owns 16
// consecutive float4 outputs; its 256 threads cut the splits into 16
// contiguous chunks (thread t: output t % 16, chunk t / 16), sum them in
// split order, and the chunk sums are combined in chunk order through LDS:
// a fixed summation order with every split read by a different thread.
__global__ __launch_bounds__(256) void wgrad_reduce4(const float4* __restrict__ part, int splits,
                                                     int64_t count4, float4* __restrict__ dw,
                                                     int accumulate) {
    __shared__ float4 red[16][16];
    const int j = threadIdx.x & 15, c = threadIdx.x >> 4;
    const int64_t i = (int64_t)blockIdx.x * 16 + j;
    const int per = (splits + 15) / 16;
    const int z0 = c * per, z1 = z0 + per < splits ? z0 + per : splits;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i < count4) {
#pragma unroll 4
        for (int z = z0; z < z1; ++z) {
            const float4 v = part[(int64_t)z * count4 + i];
            s.x += v.x;
            s.y += v.y;
            s.z += v.z;
            s.w += v.w;
        }
    }
    red[c][j] = s;
    __syncthreads();
    if (c == 0 && i < count4) {
        float4 t = accumulate ? dw[i] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            t.x += red[k][j].x;
            t.y += red[k][j].y;
            t.z += red[k][j].z;
            t.w += red[k][j].w;
        }
        dw[i] = t;
    }
}

__global__ void wgrad_reduce(const float* __restrict__ part, int splits, int64_t count,
                             float* __restrict__ dw, int accumulate) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= count) return;
    float s = accumulate ? dw[i] : 0.f;
#pragma unroll 8
    for (int z = 0; z < splits; ++z) s += part[(int64_t)z * count + i];
    dw[i] = s;
}

// dbias: stage 1 sums one segment of one (n, c) plane per block (each plane
// split into SP segments), stage 2 adds each channel's N*SP segment sums in
// order.
static int bias_segments(const ConvGeom& g) {
    const int sp = (int)ceil_div(64, g.N);
    return sp < 1 ? 1 : sp;
}

// Block (c, n * SP + segment): the sum of one segment of plane (n, c).
// Segments are multiples of 8 elements; with V % 8 == 0 every thread reads
// 8 elements per 16-byte load, four loads in flight (clamped in-segment
// addresses, out-of-segment lanes masked), else one element per load.
template <typename T>
__global__ __launch_bounds__(256) void bias_grad_part(const T* __restrict__ dy, int C, int64_t V,
                                                      int SP, float* __restrict__ part) {
    __shared__ float red[256];
    const int c = blockIdx.x, sl = blockIdx.y;  // sl = n * SP + segment
    const int n = sl / SP, seg = sl - n * SP;
    const int64_t len = ((V + SP - 1) / SP + 7) & ~(int64_t)7;
    const int64_t beg = seg * len, end = beg + len < V ? beg + len : V;
    const T* p = dy + ((int64_t)n * C + c) * V;
    float s = 0.f;
    constexpr int VEC = 16 / (int)sizeof(T);
    if (V % VEC == 0 && end > beg) {
        constexpr int64_t STEP = 256 * VEC;
        for (int64_t e0 = beg + threadIdx.x * VEC; e0 < end; e0 += 4 * STEP) {
            float v[4][VEC];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t e = e0 + u * STEP;
                vload<T, VEC>(p + (e < end ? e : end - VEC), v[u]);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const bool ok = e0 + u * STEP < end;
#pragma unroll
                for (int j = 0; j < VEC; ++j) s += ok ? v[u][j] : 0.f;
            }
        }
    } else {
        for (int64_t e = beg + threadIdx.x; e < end; e += 256) s += Elt<T>::ld(p + e);
    }
    red[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) part[(int64_t)c * gridDim.y + sl] = red[0];
}

__global__ void bias_grad_final(const float* __restrict__ part, int C, int S,
                                float* __restrict__ db, int accumulate) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    float s = accumulate ? db[c] : 0.f;
    for (int i = 0; i < S; ++i) s += part[(int64_t)c * S + i];
    db[c] = s;
}

size_t bias_grad_ws(const ConvGeom& g) {
    return (size_t)g.Co * g.N * bias_segments(g) * sizeof(float);
}

// ---------------------------------------------------------------- launchers
int wgrad_gather_splits(const ConvGeom& g) {
    const int64_t Ktot = (int64_t)g.N * g.Do * g.Ho * g.Wo;
    const int64_t tiles = ceil_div(g.Co, 64) * ceil_div((int64_t)g.Ci * g.k * g.k * g.k, 64);
    int64_t splits = ceil_div(2048, tiles);
    const int64_t max_splits = ceil_div(Ktot, 256);  // at least 256 voxels per split
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    if (splits > 4096) splits = 4096;
    return (int)splits;
}

size_t wgrad_gather_ws(const ConvGeom& g) {
    return (size_t)wgrad_gather_splits(g) * g.Co * g.Ci * g.k * g.k * g.k * sizeof(float);
}

double conv_flops(const ConvGeom& g) {
    return 2.0 * g.N * g.Co * g.Ci * (double)(g.k * g.k * g.k) * g.Do * g.Ho * g.Wo;
}

double conv_bytes(const ConvGeom& g, size_t esz) {
    return (double)esz * ((double)g.N * g.Ci * g.D * g.H * g.W +
                          (double)g.Co * g.Ci * g.k * g.k * g.k +
                          (double)g.N * g.Co * g.Do * g.Ho * g.Wo);
}

template <typename T>
static rat3d_status gather_fd(const ConvGeom& g, bool dgrad, const void* src, const void* w,
                              const float* bias, void* dst, int accumulate, hipStream_t st) {
    ProfScope ps(dgrad ? "conv_gather_dgrad" : "conv_gather_fwd", st, conv_flops(g),
                 conv_bytes(g, sizeof(T)));
    const int64_t rows = (int64_t)g.N * (dgrad ? (int64_t)g.D * g.H * g.W
                                               : (int64_t)g.Do * g.Ho * g.Wo);
    const int cols = dgrad ? g.Ci : g.Co;
    dim3 grid((unsigned)ceil_div(rows, 64), (unsigned)ceil_div(cols, 64));
    if constexpr (std::is_same<T, bf16>::value) {
        // (16-byte weight loads: K = Ci k^3 is a multiple of 8, the base must be aligned)
        if (!dgrad && !accumulate && g.Ci % 32 == 0 && g.k * g.k * g.k <= kGatherMaxTaps &&
            ((uintptr_t)w & 15u) == 0) {
            conv_gather_fwd_pipe<<<grid, 256, 0, st>>>(g, (const bf16*)src, (const bf16*)w, bias,
                                                       (bf16*)dst);
            RAT3D_LAUNCH_CHECK();
            return RAT3D_OK;
        }
    }
    if (dgrad)
        conv_gather_fd<T, true><<<grid, 256, 0, st>>>(g, (const T*)src, (const T*)w, nullptr,
                                                      (T*)dst, accumulate);
    else
        conv_gather_fd<T, false><<<grid, 256, 0, st>>>(g, (const T*)src, (const T*)w, bias,
                                                       (T*)dst, accumulate);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status conv_fwd_gather(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* w,
                             const float* bias, void* y, hipStream_t st) {
    return dt == RAT3D_BF16 ? gather_fd<bf16>(g, false, x, w, bias, y, 0, st)
                            : gather_fd<float>(g, false, x, w, bias, y, 0, st);
}

template <typename T>
static rat3d_status gather_dgrad_phase(const ConvGeom& g, const void* dy, const void* w, void* dx,
                                       int accumulate, hipStream_t st) {
    ProfScope ps("conv_gather_dgrad_s2", st, conv_flops(g), conv_bytes(g, sizeof(T)));
    // the largest class (residue 0 on every axis) sets the row grid
    const int64_t rows = (int64_t)g.N * ceil_div(g.D, g.s) * ceil_div(g.H, g.s) *
                         ceil_div(g.W, g.s);
    dim3 grid((unsigned)ceil_div(rows, 64), (unsigned)ceil_div(g.Ci, 64),
              (unsigned)(g.s * g.s * g.s));
    if constexpr (std::is_same<T, bf16>::value) {
        // class tap sets of at most (k / s + 1)^3 taps, offsets within +-127
        const int tps = g.k / g.s + 1;
        if (g.Co % 32 == 0 && tps * tps * tps <= kPhaseMaxTaps && g.k <= 127) {
            conv_gather_dgrad_phase_pipe<<<grid, 256, 0, st>>>(g, (const bf16*)dy, (const bf16*)w,
                                                               (bf16*)dx, accumulate);
            RAT3D_LAUNCH_CHECK();
            return RAT3D_OK;
        }
    }
    conv_gather_dgrad_phase<T><<<grid, 256, 0, st>>>(g, (const T*)dy, (const T*)w, (T*)dx,
                                                     accumulate);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status conv_dgrad_gather(const ConvGeom& g, rat3d_dtype dt, const void* dy, const void* w,
                               void* dx, int accumulate, hipStream_t st) {
    if (g.s > 1)  // phase-decomposed: no structurally zero products
        return dt == RAT3D_BF16 ? gather_dgrad_phase<bf16>(g, dy, w, dx, accumulate, st)
                                : gather_dgrad_phase<float>(g, dy, w, dx, accumulate, st);
    return dt == RAT3D_BF16 ? gather_fd<bf16>(g, true, dy, w, nullptr, dx, accumulate, st)
                            : gather_fd<float>(g, true, dy, w, nullptr, dx, accumulate, st);
}

rat3d_status conv_wgrad_gather(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* dy,
                               float* dw, int accumulate, void* ws, hipStream_t st) {
    const int splits = wgrad_gather_splits(g);
    const int64_t Ktot = (int64_t)g.N * g.Do * g.Ho * g.Wo;
    const int BK = dt == RAT3D_BF16 ? 32 : 16;
    const int64_t kchunk = ceil_div(ceil_div(Ktot, splits), BK) * BK;
    const int real_splits = (int)ceil_div(Ktot, kchunk);
    const int Ncols = g.Ci * g.k * g.k * g.k;
    dim3 grid((unsigned)ceil_div(g.Co, 64), (unsigned)ceil_div(Ncols, 64), (unsigned)real_splits);
    float* part = (float*)ws;
    {
    ProfScope ps("conv_gather_wgrad", st, conv_flops(g),
                 conv_bytes(g, dt == RAT3D_BF16 ? 2 : 4));
    if (dt == RAT3D_BF16)
        conv_gather_wgrad<bf16><<<grid, 256, 0, st>>>(g, (const bf16*)x, (const bf16*)dy, part,
                                                      kchunk);
    else
        conv_gather_wgrad<float><<<grid, 256, 0, st>>>(g, (const float*)x, (const float*)dy,
                                                       part, kchunk);
    RAT3D_LAUNCH_CHECK();
    }
    const int64_t count = (int64_t)g.Co * Ncols;
    ProfScope ps("wgrad_reduce", st, 0.0, 4.0 * count * (real_splits + 1 + accumulate));
    return wgrad_reduce_launch(part, real_splits, count, dw, accumulate, st);
}

rat3d_status wgrad_reduce_launch(const float* part, int splits, int64_t count, float* dw,
                                 int accumulate, hipStream_t st) {
    if (count % 4 == 0 && ((uintptr_t)dw & 15u) == 0 && ((uintptr_t)part & 15u) == 0)
        wgrad_reduce4<<<(unsigned)ceil_div(count / 4, 16), 256, 0, st>>>(
            (const float4*)part, splits, count / 4, (float4*)dw, accumulate);
    else
        wgrad_reduce<<<(unsigned)ceil_div(count, 256), 256, 0, st>>>(part, splits, count, dw,
                                                                     accumulate);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status conv_bias_grad(const ConvGeom& g, rat3d_dtype dt, const void* dy, float* db,
                            int accumulate, void* ws, hipStream_t st) {
    const int64_t Vo = (int64_t)g.Do * g.Ho * g.Wo;
    float* part = (float*)ws;
    ProfScope ps("bias_grad", st, 0.0, (dt == RAT3D_BF16 ? 2.0 : 4.0) * g.N * g.Co * Vo);
    const int SP = bias_segments(g);
    const dim3 grid(g.Co, g.N * SP);
    if (dt == RAT3D_BF16)
        bias_grad_part<bf16><<<grid, 256, 0, st>>>((const bf16*)dy, g.Co, Vo, SP, part);
    else
        bias_grad_part<float><<<grid, 256, 0, st>>>((const float*)dy, g.Co, Vo, SP, part);
    RAT3D_LAUNCH_CHECK();
    bias_grad_final<<<(unsigned)ceil_div(g.Co, 64), 64, 0, st>>>(part, g.Co, g.N * SP, db,
                                                                 accumulate);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

// One wave per channel: lane l adds partials l, l + 64, ... in turn, then an
// xor butterfly (a fixed order for a given S).
__global__ __launch_bounds__(64) void bias_sum_wave(const float* __restrict__ part, int S,
                                                    float* __restrict__ db, int accumulate) {
    const int c = blockIdx.x, lane = threadIdx.x;
    const float* p = part + (int64_t)c * S;
    float s = 0.f;
    for (int i = lane; i < S; i += 64) s += p[i];
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
    if (lane == 0) db[c] = accumulate ? db[c] + s : s;
}

rat3d_status bias_grad_from_partials(const float* part, int C, int S, float* db, int accumulate,
                                     hipStream_t st) {
    bias_sum_wave<<<(unsigned)C, 64, 0, st>>>(part, S, db, accumulate);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

}  // namespace rat3d
