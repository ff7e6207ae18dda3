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
// reads.  A workgroup walks a range of bricks with the next brick's dy and
// input loads in flight while the current one is multiplied.
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
    int nbricks;
    int bpr;
};
}  // namespace

__global__ __launch_bounds__(256, 2) void stem_wgrad_k(StemWg a) {
    // xs: parity plane p holds brick columns 2c + p, rows of kGHalf columns;
    // shift 1 is the same plane moved left by one column.  dys[ct][step][lane]:
    // the A operand of each step in MFMA lane order, lane = kg * 16 + li holding
    // the 8 voxels (d0 + dl, h0 + 2 (step % 4) + (kg >> 1), w0 + 8 (kg & 1) ..)
    // of channel ct * 16 + li (dl = step / 4)
    constexpr int kSteps = kGD * kGH / 2;
    // plane (parity p, shift s) starts at (2 p + s) * kGPlane elements: the
    // 112-byte pad spreads the B reads of one instruction, whose lanes hit
    // all four planes, over the LDS banks
    constexpr int kGPlane = kGBD * kGBH * kGHalf + 56;
    __shared__ __align__(16) bf16 xs[4 * kGPlane];
    __shared__ __align__(16) uint4 dys[2 * kSteps * 64];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar branches
    __builtin_assume(tid < 256);
    const int li = lane & 15, kg = lane >> 4;
    const int hl_l = kg >> 1, wl = (kg & 1) * 8;
    const int b_beg = blockIdx.x * a.bpr;
    const int b_end = b_beg + a.bpr < a.nbricks ? b_beg + a.bpr : a.nbricks;
    const int64_t HW = (int64_t)a.H * a.W, Vo = (int64_t)a.Do * a.Ho * a.Wo;

    // One brick's staging registers: its dy units (thread tid fills the dys
    // slots tid + 256 i: consecutive lanes, consecutive 16-byte slots) and
    // its input items.  Input staging (W % 8 == 0): brick column c is input
    // column a0 + 5 + c (a0 = bw - 5, a multiple of 8).  With G the row's
    // dwords from a0, plane 0 column cc = high half of G[cc + 2], plane 1
    // column cc = low half of G[cc + 3]; the shifted copies start one column
    // later.  An item (row, k) builds dwords 4k .. 4k + 3 of the four plane
    // copies from the three aligned 16-byte groups G[8k .. 8k + 11], of which
    // G[8k] and G[8k + 1] are not used.
    constexpr int NDU = kSCo * kGD * kGH * 2 / 256;   // dy units per thread (4)
    constexpr int NIT = kGBD * kGBH * 3;
    constexpr int NI = (NIT + 255) / 256;             // items per thread, at most
    struct Stage {
        uint4 dv[NDU];
        uint2 gv0[NI];
        uint4 gv[NI][2];
    };
    // Buffer loads of the sample's dy and input volumes: an offset past the
    // end (voxels outside the map, padding) reads zeros.
    auto issue = [&](int b, Stage& S) {
        const int twi = b % a.tw;
        int r = b / a.tw;
        const int thi = r % a.th;
        r /= a.th;
        const int tdi = r % a.td;
        const int n = r / a.td;
        const int d0 = tdi * kGD, h0 = thi * kGH, w0 = twi * kGW;
        const int bd = d0 * kSS - kSP, bh = h0 * kSS - kSP, bw = w0 * kSS - kSP;
        const __amdgpu_buffer_rsrc_t dyr =
            buf_rsrc_u(a.dy + (int64_t)n * kSCo * Vo, (uint32_t)(kSCo * Vo * 2));
        const __amdgpu_buffer_rsrc_t xr =
            buf_rsrc_u(a.x + (int64_t)n * a.D * HW, (uint32_t)(a.D * HW * 2));
#pragma unroll
        for (int i = 0; i < NDU; ++i) {
            const int u = tid + 256 * i;
            const int ul = u & 63, step = (u >> 6) & 7, co = (u >> 9) * 16 + (ul & 15);
            const int ukg = ul >> 4, dl = step >> 2, hl = (step & 3) * 2 + (ukg >> 1);
            const int d = d0 + dl, h = h0 + hl, w = w0 + 8 * (ukg & 1);
            const bool ok = d < a.Do && h < a.Ho && w + 8 <= a.Wo;
            const uint32_t vo =
                ok ? (uint32_t)((co * Vo + ((int64_t)d * a.Ho + h) * a.Wo + w) * 2) : 0x80000000u;
            S.dv[i] = buf_ld16(dyr, vo, 0);
        }
        const int a0 = bw - 5;
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
                const uint32_t xo = ok ? (uint32_t)((d * HW + h * a.W + c0) * 2) : 0x80000000u;
                if (q == 0) S.gv0[j] = buf_ld8(xr, xo, 8);
                else S.gv[j][q - 1] = buf_ld16(xr, xo, 0);
            }
        }
    };
    // The staged brick into LDS (no brick coordinates needed).
    auto commit = [&](const Stage& S) {
#pragma unroll
        for (int i = 0; i < NDU; ++i) dys[tid + 256 * i] = S.dv[i];
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int it = tid + 256 * j;
            if (it >= NIT) continue;
            const int k = it % 3, row = it / 3;
            const uint32_t g[12] = {0u, 0u, S.gv0[j].x, S.gv0[j].y,
                                    S.gv[j][0].x, S.gv[j][0].y, S.gv[j][0].z, S.gv[j][0].w,
                                    S.gv[j][1].x, S.gv[j][1].y, S.gv[j][1].z, S.gv[j][1].w};
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
            bf16* const xr = &xs[row * kGHalf + 8 * k];
            *reinterpret_cast<uint4*>(xr) = make_uint4(p0[0], p0[1], p0[2], p0[3]);
            *reinterpret_cast<uint4*>(xr + 2 * kGPlane) = make_uint4(p1[0], p1[1], p1[2], p1[3]);
            *reinterpret_cast<uint4*>(xr + kGPlane) = make_uint4(s0[0], s0[1], s0[2], s0[3]);
            *reinterpret_cast<uint4*>(xr + 3 * kGPlane) = make_uint4(s1[0], s1[1], s1[2], s1[3]);
        }
    };

    f32x4 acc[kTilesPerWave][2];
#pragma unroll
    for (int j = 0; j < kTilesPerWave; ++j) {
        acc[j][0] = f32x4{0.f, 0.f, 0.f, 0.f};
        acc[j][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    auto compute = [&]() {
#pragma unroll
        for (int s = 0; s < kSteps; ++s) {
            const int dl = s / (kGH / 2);
            const int hl = (s % (kGH / 2)) * 2 + hl_l;
            F16B av[2];
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) av[ct].u = dys[(ct * kSteps + s) * 64 + lane];
            // tiles wave + 4 j: all exist for j < kTilesPerWave - 1, the last
            // only for the waves below kTapTiles % 4 (one wave-uniform branch)
            const int nj = wave + 4 * (kTilesPerWave - 1) < kTapTiles ? kTilesPerWave
                                                                     : kTilesPerWave - 1;
#pragma unroll
            for (int j = 0; j < kTilesPerWave; ++j) {
                if (j == kTilesPerWave - 1 && j >= nj) break;
                const int tile = wave + 4 * j;
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
                    const bf16* src = &xs[((kwc & 1) * 2 + sh) * kGPlane +
                                          ((dl * kSS + kd) * kGBH + hl * kSS + kh) * kGHalf +
                                          start - sh];
#pragma unroll
                    for (int q = 0; q < 4; ++q) bv.w[q] = reinterpret_cast<const uint32_t*>(src)[q];
                }
#pragma unroll
                for (int ct = 0; ct < 2; ++ct)
                    acc[j][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[ct].b, bv.b,
                                                                        acc[j][ct], 0, 0, 0);
            }
        }
    };

    // Software pipeline: brick b + 1's loads are issued right after brick b
    // is written to LDS, so their round trip overlaps brick b's MFMAs.
    Stage S;
    if (b_beg < b_end) issue(b_beg, S);
    for (int b = b_beg; b < b_end; ++b) {
        __syncthreads();  // every wave is done reading the previous brick
        commit(S);
        if (b + 1 < b_end) issue(b + 1, S);
        __syncthreads();
        compute();
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
    int64_t r = 512;  // two workgroups per CU
    if (r > nbricks) r = nbricks;
    return (int)(r < 1 ? 1 : r);
}

static int64_t stem_bricks(const ConvGeom& g) {
    return (int64_t)g.N * ceil_div(g.Do, kGD) * ceil_div(g.Ho, kGH) * ceil_div(g.Wo, kGW);
}

bool stem_wgrad_ok(const ConvGeom& g, rat3d_dtype dt) {
    // one sample's dy and input volumes are addressed with 32-bit byte offsets
    return stem_ok(g, dt) && g.Wo % 8 == 0 &&
           (int64_t)kSCo * g.Do * g.Ho * g.Wo * 2 < (1LL << 31) &&
           (int64_t)g.D * g.H * g.W * 2 < (1LL << 31) && stem_bricks(g) < (1LL << 31);
}

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
