// The stem convolution: one input channel, cubic kernel 7, stride 2, pad 3
// (bf16).  With a single input channel the GEMM K index is the tap alone, so
// the channel-chunked brick kernels do not apply.
//
// Forward: a workgroup computes 4 x 8 x 16 output voxels for 32 output
// channels.  K is ordered (kd, kh, kw) with kw padded from 7 to 8, so the
// eight K values of one MFMA operand row are eight consecutive input columns
// of one (kd, kh) row: columns 2i .. 2i+7 of the input brick for output
// column i, four 4-byte LDS reads.  Padding taps (kw = 7, and (kd, kh) rows
// 49..51 of the last K step) have zero weights.  The weights are re-laid in
// MFMA lane order once per launch and copied into LDS with the brick: every
// staging load of a workgroup is issued before the first LDS store, so a
// workgroup waits for one global round trip, and three workgroups share a
// CU.
//
// Weight gradient: rows = output channels, columns = padded taps, K = output
// voxels.  The A operand is dy (8 consecutive output voxels of one channel),
// staged in LDS in MFMA lane order; the B operand needs input columns
// 2w - 3 + kw at stride 2, so the input brick is stored split by column
// parity, each parity plane twice (shifted by one element) so that the 8
// values start on a 4-byte boundary and load as four aligned 4-byte LDS
// reads.  Each brick's dy and input loads are all issued before the barrier
// that frees the LDS, and three workgroups share a CU.
#include "common.hpp"
#include "kernels.hpp"
#include "prof.hpp"

namespace rat3d {

namespace {
union F16B {
    uint4 u;
    uint2 h[2];
    uint32_t w[4];
    bf16x8 b;
};

constexpr int kSK = 7, kSS = 2, kSP = 3;          // kernel, stride, pad
constexpr int kSRows = kSK * kSK;                 // (kd, kh) rows
constexpr int kSRowsPad = 52;                     // 13 K steps x 4 rows
constexpr int kSCo = 32;                          // output channels handled

// forward tile and brick
constexpr int kFD = 4, kFH = 8, kFW = 16;
constexpr int kFBD = (kFD - 1) * kSS + kSK;       // 13
constexpr int kFBH = (kFH - 1) * kSS + kSK;       // 21
constexpr int kFBW = 40;                          // >= (16-1)*2 + 8 = 38 columns, 80-byte rows
}  // namespace

// wp[ks][ct][lane][8], the B operands in MFMA lane order: lane = kg * 16 + li
// holds w[co][0][kd][kh][kw] for co = ct * 16 + li, row r = kd * 7 + kh =
// 4 ks + kg and kw = 0 .. 7; zero for kw = 7 and rows past 48
constexpr int kSKSteps = kSRowsPad / 4;           // 13 K steps
constexpr int kSWUnits = kSKSteps * 2 * 64;       // 16-byte units of wp
__global__ void stem_prep_weights(const bf16* __restrict__ w, bf16* __restrict__ wp) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= kSWUnits * 8) return;
    const int kw = i & 7, lane = (i >> 3) & 63, ct = (i >> 9) & 1, ks = i >> 10;
    const int co = ct * 16 + (lane & 15), r = ks * 4 + (lane >> 4);
    bf16 v = 0;
    if (kw < kSK && r < kSRows) v = w[(co * kSRows + r) * kSK + kw];
    wp[i] = v;
}

__global__ __launch_bounds__(256, 3) void stem_fwd_k(const bf16* __restrict__ x,
                                                     const bf16* __restrict__ wp,
                                                     bf16* __restrict__ y, int N, int D, int H,
                                                     int W, int Do, int Ho, int Wo, int td,
                                                     int th, int tw) {
    constexpr int NWU = (kSWUnits + 255) / 256;       // weight units per thread
    constexpr int NCH = kFBW / 8;                     // 16-byte chunks per brick row (5)
    constexpr int NIT = kFBD * kFBH * NCH;            // staging items (1365)
    constexpr int NI = (NIT + 255) / 256;             // items per thread
    // rows past kFBD * kFBH take the stores of items past NIT and are never read
    __shared__ __align__(16) bf16 brick[(NI * 256 + NCH - 1) / NCH * kFBW];
    __shared__ __align__(16) uint4 wl[NWU * 256];     // units past kSWUnits: unused
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    __builtin_assume(tid < 256);
    const int li = lane & 15, kg = lane >> 4;
    int L = blockIdx.x;
    const int twi = L % tw;
    L /= tw;
    const int thi = L % th;
    L /= th;
    const int tdi = L % td;
    const int n = L / td;
    const int d0 = tdi * kFD, h0 = thi * kFH, w0 = twi * kFW;
    const int bd = d0 * kSS - kSP, bh = h0 * kSS - kSP, bw = w0 * kSS - kSP;
    const int64_t HW = (int64_t)H * W;
    const bf16* xp = x + (int64_t)n * D * HW;

    // Staging (W % 8 == 0): brick column c is input column bw + c with
    // bw = 2 w0 - 3 = a0 + 5, a0 a multiple of 8.  A brick row is five
    // 16-byte chunks; chunk k holds input dwords G[4k + 2 ..] moved by one
    // bf16 (G = the row's dwords from a0).  Each item loads the two aligned
    // 16-byte groups that cover it (rows or groups outside the volume load
    // from a clamped address and are zeroed).  The weight units and all items
    // of a thread are loaded before anything is stored.
    {
        const int a0 = bw - 5;
        const int64_t plane = (int64_t)D * HW;
        uint4 wv[NWU];
#pragma unroll
        for (int i = 0; i < NWU; ++i) {
            const int u = tid + 256 * i;
            wv[i] = reinterpret_cast<const uint4*>(wp)[u < kSWUnits ? u : 0];
        }
        uint4 gv[NI][2];
        uint32_t okm = 0;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int it = tid + 256 * j;
            const int k = it % NCH, r = it / NCH;
            const int hh = r % kFBH, dd = r / kFBH;
            const int d = bd + dd, h = bh + hh;
            const bool rok = it < NIT && (unsigned)d < (unsigned)D && (unsigned)h < (unsigned)H;
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const int c0 = a0 + 8 * (k + q);
                const bool ok = rok && c0 >= 0 && c0 < W;
                const int64_t off = ok ? (int64_t)d * HW + (int64_t)h * W + c0 : 0;
                gv[j][q] = *reinterpret_cast<const uint4*>(xp + (off < plane ? off : 0));
                okm |= (ok ? 1u : 0u) << (2 * j + q);
            }
        }
        __builtin_amdgcn_sched_barrier(0);  // every load above is issued before any is used
#pragma unroll
        for (int i = 0; i < NWU; ++i) wl[tid + 256 * i] = wv[i];
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int it = tid + 256 * j;
            const int k = it % NCH, r = it / NCH;
            uint32_t g[8];
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const bool ok = (okm >> (2 * j + q)) & 1u;
                g[4 * q + 0] = ok ? gv[j][q].x : 0u;
                g[4 * q + 1] = ok ? gv[j][q].y : 0u;
                g[4 * q + 2] = ok ? gv[j][q].z : 0u;
                g[4 * q + 3] = ok ? gv[j][q].w : 0u;
            }
            // brick dword m (columns 2m, 2m + 1) = high half of G[m + 2], low half of G[m + 3]
            uint32_t o[4];
#pragma unroll
            for (int m = 0; m < 4; ++m) o[m] = __builtin_amdgcn_alignbit(g[m + 3], g[m + 2], 16);
            *reinterpret_cast<uint4*>(&brick[r * kFBW + 8 * k]) = make_uint4(o[0], o[1], o[2], o[3]);
        }
    }
    __syncthreads();

    f32x4 acc[8][2];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        acc[i][0] = f32x4{0.f, 0.f, 0.f, 0.f};
        acc[i][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    // operand of output column li: brick columns 2 li .. 2 li + 7, which start
    // on a 4-byte boundary (rows are 80 bytes)
#pragma unroll
    for (int ks = 0; ks < kSKSteps; ++ks) {
        const int r = ks * 4 + kg;
        F16B b[2];
#pragma unroll
        for (int ct = 0; ct < 2; ++ct) b[ct].u = wl[(ks * 2 + ct) * 64 + lane];
        const int rr = r < kSRows ? r : kSRows - 1;  // padding rows: any valid row, zero weights
        const int kd = rr / kSK, kh = rr - kd * kSK;
#pragma unroll
        for (int rw = 0; rw < 8; ++rw) {
            const int dd = wave * kSS + kd, hh = rw * kSS + kh;
            const uint32_t* src =
                reinterpret_cast<const uint32_t*>(&brick[(dd * kFBH + hh) * kFBW + 2 * li]);
            F16B a;
#pragma unroll
            for (int q = 0; q < 4; ++q) a.w[q] = src[q];
#pragma unroll
            for (int ct = 0; ct < 2; ++ct)
                acc[rw][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.b, b[ct].b, acc[rw][ct],
                                                                     0, 0, 0);
        }
    }

    const int d = d0 + wave;
    if (d >= Do) return;
    const int64_t V = (int64_t)Do * Ho * Wo;
    const bool full = (w0 + kFW <= Wo) && (Wo % 4 == 0);
#pragma unroll
    for (int rw = 0; rw < 8; ++rw) {
        const int h = h0 + rw;
        if (h >= Ho) continue;
#pragma unroll
        for (int ct = 0; ct < 2; ++ct) {
            const int co = ct * 16 + li;
            const int w = w0 + 4 * kg;
            bf16* q = y + ((int64_t)n * kSCo + co) * V + ((int64_t)d * Ho + h) * Wo + w;
            if (full) {
                *reinterpret_cast<uint2*>(q) =
                    make_uint2(pack_bf16x2(acc[rw][ct][0], acc[rw][ct][1]),
                               pack_bf16x2(acc[rw][ct][2], acc[rw][ct][3]));
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (w + e < Wo) q[e] = f2bf(acc[rw][ct][e]);
            }
        }
    }
}

// ---------------------------------------------------------------- weight gradient
namespace {
constexpr int kGD = 2, kGH = 8, kGW = 16;          // output voxels per brick (256)
constexpr int kGBD = (kGD - 1) * kSS + kSK;        // 9
constexpr int kGBH = (kGH - 1) * kSS + kSK;        // 21
constexpr int kGHalf = 24;                         // parity-plane columns (>= 19 + 3 + pad)
constexpr int kTapTiles = (kSRows * 8 + 15) / 16;  // 25 tiles of 16 padded taps
constexpr int kTilesPerWave = (kTapTiles + 3) / 4; // 7

struct StemWg {
    const bf16* x;
    const bf16* dy;
    float* part;  // [ranges][32][kSRows * 8]
    int N, D, H, W, Do, Ho, Wo;
    int td, th, tw;
    int64_t nbricks;
    int bpr;
};
}  // namespace

__global__ __launch_bounds__(256, 3) void stem_wgrad_k(StemWg a) {
    // xs[parity][shift][row][col]: parity plane p holds brick columns 2c + p;
    // shift 1 is the same plane moved left by one column.  dys[ct][step][lane]:
    // the A operand of each step in MFMA lane order, lane = kg * 16 + li holding
    // the 8 voxels (d0 + dl, h0 + 2 (step % 4) + (kg >> 1), w0 + 8 (kg & 1) ..)
    // of channel ct * 16 + li (dl = step / 4)
    constexpr int kSteps = kGD * kGH / 2;
    __shared__ __align__(16) bf16 xs[2][2][kGBD * kGBH][kGHalf];
    __shared__ __align__(16) uint4 dys[2 * kSteps * 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    __builtin_assume(tid < 256);
    const int li = lane & 15, kg = lane >> 4;
    const int hl_l = kg >> 1, wl = (kg & 1) * 8;
    const int64_t b_beg = (int64_t)blockIdx.x * a.bpr;
    const int64_t b_end = b_beg + a.bpr < a.nbricks ? b_beg + a.bpr : a.nbricks;
    const int64_t HW = (int64_t)a.H * a.W, Vo = (int64_t)a.Do * a.Ho * a.Wo;

    f32x4 acc[kTilesPerWave][2];
#pragma unroll
    for (int j = 0; j < kTilesPerWave; ++j) {
        acc[j][0] = f32x4{0.f, 0.f, 0.f, 0.f};
        acc[j][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    for (int64_t b = b_beg; b < b_end; ++b) {
        const int twi = (int)(b % a.tw);
        int64_t r = b / a.tw;
        const int thi = (int)(r % a.th);
        r /= a.th;
        const int tdi = (int)(r % a.td);
        const int n = (int)(r / a.td);
        const int d0 = tdi * kGD, h0 = thi * kGH, w0 = twi * kGW;
        const int bd = d0 * kSS - kSP, bh = h0 * kSS - kSP, bw = w0 * kSS - kSP;
        const bf16* xp = a.x + (int64_t)n * a.D * HW;
        // Every load of the brick is issued before the barrier that ends the
        // previous brick's MFMAs, so the round trip overlaps them.
        // dy: 32 channels x 2 depths x 8 rows x two 8-voxel halves, unit
        // u = ((co * 2 + dl) * 8 + hl) * 2 + half; outside the map: zero (the
        // load reads the plane's first voxels)
        constexpr int NDU = kSCo * kGD * kGH * 2 / 256;   // dy units per thread (4)
        uint4 dv[NDU];
        uint32_t dokm = 0;
#pragma unroll
        for (int i = 0; i < NDU; ++i) {
            const int u = tid + 256 * i;
            const int half = u & 1, hl = (u >> 1) & 7, dl = (u >> 4) & 1, co = u >> 5;
            const int d = d0 + dl, h = h0 + hl, w = w0 + 8 * half;
            const bool ok = d < a.Do && h < a.Ho && w + 8 <= a.Wo;
            const int64_t vo = ok ? ((int64_t)d * a.Ho + h) * a.Wo + w : 0;
            dv[i] = *reinterpret_cast<const uint4*>(a.dy + ((int64_t)n * kSCo + co) * Vo + vo);
            dokm |= (ok ? 1u : 0u) << i;
        }
        // Input staging (W % 8 == 0): brick column c is input column a0 + 5 + c
        // (a0 = bw - 5, a multiple of 8).  With G the row's dwords from a0,
        // plane 0 column cc = high half of G[cc + 2], plane 1 column cc = low
        // half of G[cc + 3]; the shifted copies start one column later.  An
        // item (row, k) builds dwords 4k .. 4k + 3 of the four plane copies
        // from the three aligned 16-byte groups G[8k .. 8k + 11] (rows or
        // groups outside the volume: clamped address, zeroed).
        const int a0 = bw - 5;
        constexpr int NIT = kGBD * kGBH * 3;
        constexpr int NI = (NIT + 255) / 256;             // items per thread, at most
        const int64_t plane = (int64_t)a.D * HW;
        // G[8k], G[8k + 1] are not used: the first group loads its upper 8 bytes
        uint2 gv0[NI];
        uint4 gv[NI][2];
        uint32_t okm = 0;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int it = tid + 256 * j;
            const int k = it % 3, row = it / 3;
            const int hh = row % kGBH, dd = row / kGBH;
            const int d = bd + dd, h = bh + hh;
            const bool rok = it < NIT && (unsigned)d < (unsigned)a.D && (unsigned)h < (unsigned)a.H;
#pragma unroll
            for (int q = 0; q < 3; ++q) {
                const int c0 = a0 + 8 * (2 * k + q);
                const bool ok = rok && c0 >= 0 && c0 < a.W;
                const int64_t off = ok ? (int64_t)d * HW + (int64_t)h * a.W + c0 : 0;
                const bf16* src = xp + (off < plane ? off : 0);
                if (q == 0) gv0[j] = reinterpret_cast<const uint2*>(src)[1];
                else gv[j][q - 1] = *reinterpret_cast<const uint4*>(src);
                okm |= (ok ? 1u : 0u) << (3 * j + q);
            }
        }
        __builtin_amdgcn_sched_barrier(0);  // every load above is issued before any is used
        __syncthreads();
#pragma unroll
        for (int i = 0; i < NDU; ++i) {
            const int u = tid + 256 * i;
            const int half = u & 1, hl = (u >> 1) & 7, dl = (u >> 4) & 1, co = u >> 5;
            const int step = dl * 4 + (hl >> 1), ul = ((hl & 1) * 2 + half) * 16 + (co & 15);
            dys[((co >> 4) * kSteps + step) * 64 + ul] =
                (dokm >> i) & 1u ? dv[i] : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int it = tid + 256 * j;
            if (it >= NIT) continue;
            const int k = it % 3, row = it / 3;
            uint32_t g[12];
            {
                const bool ok = okm >> (3 * j) & 1u;
                g[0] = g[1] = 0u;
                g[2] = ok ? gv0[j].x : 0u;
                g[3] = ok ? gv0[j].y : 0u;
            }
#pragma unroll
            for (int q = 1; q < 3; ++q) {
                const bool ok = (okm >> (3 * j + q)) & 1u;
                g[4 * q + 0] = ok ? gv[j][q - 1].x : 0u;
                g[4 * q + 1] = ok ? gv[j][q - 1].y : 0u;
                g[4 * q + 2] = ok ? gv[j][q - 1].z : 0u;
                g[4 * q + 3] = ok ? gv[j][q - 1].w : 0u;
            }
            // plane dword m = 4k + j uses G[2m + 2 .. 2m + 5] = g[2j + 2 .. 2j + 5]
            uint32_t p0[4], p1[4], s0[4], s1[4];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const uint32_t a2 = g[2 * m + 2], a3 = g[2 * m + 3], a4 = g[2 * m + 4],
                               a5 = g[2 * m + 5];
                p0[m] = __builtin_amdgcn_perm(a3, a2, 0x07060302u);  // hi(a2) | hi(a3) << 16
                p1[m] = __builtin_amdgcn_perm(a4, a3, 0x05040100u);  // lo(a3) | lo(a4) << 16
                s0[m] = __builtin_amdgcn_perm(a4, a3, 0x07060302u);  // hi(a3) | hi(a4) << 16
                s1[m] = __builtin_amdgcn_perm(a5, a4, 0x05040100u);  // lo(a4) | lo(a5) << 16
            }
            *reinterpret_cast<uint4*>(&xs[0][0][row][8 * k]) = make_uint4(p0[0], p0[1], p0[2], p0[3]);
            *reinterpret_cast<uint4*>(&xs[1][0][row][8 * k]) = make_uint4(p1[0], p1[1], p1[2], p1[3]);
            *reinterpret_cast<uint4*>(&xs[0][1][row][8 * k]) = make_uint4(s0[0], s0[1], s0[2], s0[3]);
            *reinterpret_cast<uint4*>(&xs[1][1][row][8 * k]) = make_uint4(s1[0], s1[1], s1[2], s1[3]);
        }
        __syncthreads();
#pragma unroll
        for (int s = 0; s < kSteps; ++s) {
            const int dl = s / (kGH / 2);
            const int hl = (s % (kGH / 2)) * 2 + hl_l;
            F16B av[2];
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) av[ct].u = dys[(ct * kSteps + s) * 64 + lane];
#pragma unroll
            for (int j = 0; j < kTilesPerWave; ++j) {
                const int tile = wave + 4 * j;
                if (tile >= kTapTiles) continue;
                // this lane's B column: padded tap t = tile*16 + li
                const int t = tile * 16 + li;
                const int rrow = t >> 3, kw = t & 7;
                // padding taps (kw = 7, rows past 49) read a valid tap; their
                // sums are never stored
                F16B bv;
                {
                    const int rr = rrow < kSRows ? rrow : kSRows - 1;
                    const int kwc = kw < kSK ? kw : kSK - 1;
                    const int kd = rr / kSK, kh = rr - kd * kSK;
                    // input column (brick) for output column wl + i: 2*(wl + i) + kw
                    // = parity kw & 1, plane column wl + i + (kw >> 1)
                    const int start = wl + (kwc >> 1);
                    const int sh = start & 1;
                    const bf16* src =
                        &xs[kwc & 1][sh][(dl * kSS + kd) * kGBH + hl * kSS + kh][start - sh];
#pragma unroll
                    for (int q = 0; q < 4; ++q) bv.w[q] = reinterpret_cast<const uint32_t*>(src)[q];
                }
#pragma unroll
                for (int ct = 0; ct < 2; ++ct)
                    acc[j][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[ct].b, bv.b,
                                                                        acc[j][ct], 0, 0, 0);
            }
        }
    }

    float* out = a.part + (int64_t)blockIdx.x * kSCo * kSRows * 8;
#pragma unroll
    for (int j = 0; j < kTilesPerWave; ++j) {
        const int tile = wave + 4 * j;
        if (tile >= kTapTiles) continue;
        const int t = tile * 16 + li;
        if ((t >> 3) >= kSRows) continue;
#pragma unroll
        for (int ct = 0; ct < 2; ++ct)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                out[(ct * 16 + 4 * kg + e) * kSRows * 8 + t] = acc[j][ct][e];
    }
}

// part is [ranges][32][49*8]; dw is [32][1][7][7][7] (padding column kw = 7
// dropped).  A block owns 16 consecutive outputs; its 256 threads cut the
// ranges into 16 contiguous chunks (thread t: output t % 16, chunk t / 16),
// sum them in range order, and the chunk sums are combined in chunk order.
__global__ __launch_bounds__(256) void stem_wgrad_reduce(const float* __restrict__ part,
                                                         int ranges, float* __restrict__ dw,
                                                         int accumulate) {
    __shared__ float red[16][16];
    const int j = threadIdx.x & 15, c = threadIdx.x >> 4;
    const int i = blockIdx.x * 16 + j;
    const bool live = i < kSCo * kSRows * kSK;
    const int kw = i % kSK, r = (i / kSK) % kSRows, co = i / (kSK * kSRows);
    const int64_t src = (int64_t)co * kSRows * 8 + r * 8 + kw;
    const int per = (ranges + 15) / 16;
    const int z0 = c * per, z1 = z0 + per < ranges ? z0 + per : ranges;
    float s = 0.f;
    if (live) {
#pragma unroll 4
        for (int z = z0; z < z1; ++z) s += part[(int64_t)z * kSCo * kSRows * 8 + src];
    }
    red[c][j] = s;
    __syncthreads();
    if (c == 0 && live) {
        float t = accumulate ? dw[i] : 0.f;
#pragma unroll
        for (int k = 0; k < 16; ++k) t += red[k][j];
        dw[i] = t;
    }
}

bool stem_ok(const ConvGeom& g, rat3d_dtype dt) {
    return dt == RAT3D_BF16 && g.Ci == 1 && g.Co == kSCo && g.k == kSK && g.s == kSS &&
           g.p == kSP && g.W % 8 == 0;
}

size_t stem_fwd_ws() { return (size_t)kSCo * kSRowsPad * 8 * 2; }

static int stem_ranges(int64_t nbricks) {
    int64_t r = 768;  // three workgroups per CU
    if (r > nbricks) r = nbricks;
    return (int)(r < 1 ? 1 : r);
}

static int64_t stem_bricks(const ConvGeom& g) {
    return (int64_t)g.N * ceil_div(g.Do, kGD) * ceil_div(g.Ho, kGH) * ceil_div(g.Wo, kGW);
}

bool stem_wgrad_ok(const ConvGeom& g, rat3d_dtype dt) { return stem_ok(g, dt) && g.Wo % 8 == 0; }

size_t stem_wgrad_ws(const ConvGeom& g) {
    return (size_t)stem_ranges(stem_bricks(g)) * kSCo * kSRows * 8 * sizeof(float);
}

rat3d_status conv_fwd_stem(const ConvGeom& g, const void* x, const void* w, void* y, void* ws,
                           hipStream_t st) {
    bf16* wp = (bf16*)ws;
    stem_prep_weights<<<(unsigned)ceil_div(kSCo * kSRowsPad * 8, 256), 256, 0, st>>>(
        (const bf16*)w, wp);
    RAT3D_LAUNCH_CHECK();
    const int td = (int)ceil_div(g.Do, kFD), th = (int)ceil_div(g.Ho, kFH),
              tw = (int)ceil_div(g.Wo, kFW);
    ProfScope ps("conv_stem_fwd", st, conv_flops(g), conv_bytes(g, 2));
    stem_fwd_k<<<(unsigned)((int64_t)g.N * td * th * tw), 256, 0, st>>>(
        (const bf16*)x, wp, (bf16*)y, g.N, g.D, g.H, g.W, g.Do, g.Ho, g.Wo, td, th, tw);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status conv_wgrad_stem(const ConvGeom& g, const void* x, const void* dy, float* dw,
                             int accumulate, void* ws, hipStream_t st) {
    StemWg a;
    a.x = (const bf16*)x;
    a.dy = (const bf16*)dy;
    a.part = (float*)ws;
    a.N = g.N;
    a.D = g.D;
    a.H = g.H;
    a.W = g.W;
    a.Do = g.Do;
    a.Ho = g.Ho;
    a.Wo = g.Wo;
    a.td = (int)ceil_div(g.Do, kGD);
    a.th = (int)ceil_div(g.Ho, kGH);
    a.tw = (int)ceil_div(g.Wo, kGW);
    a.nbricks = stem_bricks(g);
    const int R = stem_ranges(a.nbricks);
    a.bpr = (int)ceil_div(a.nbricks, R);
    const int Rreal = (int)ceil_div(a.nbricks, a.bpr);
    {
        ProfScope ps("conv_stem_wgrad", st, conv_flops(g), conv_bytes(g, 2));
        stem_wgrad_k<<<(unsigned)Rreal, 256, 0, st>>>(a);
        RAT3D_LAUNCH_CHECK();
    }
    ProfScope ps("wgrad_reduce", st, 0.0, 4.0 * kSCo * kSRows * 8 * (Rreal + 1 + accumulate));
    stem_wgrad_reduce<<<(unsigned)ceil_div(kSCo * kSRows * kSK, 16), 256, 0, st>>>(a.part, Rreal,
                                                                                  dw, accumulate);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

}  // namespace rat3d
