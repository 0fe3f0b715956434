// Dense baseline: the matrix-multiplication formulation of convolution
// (Sec. "Sparse Convolution", Fig. 3), M_K [K x RSC] * M_I [RSC x HoWo] =
// M_O [K x HoWo], with the batch appended as extra columns of M_I.
//
// M_I has row (c, r, s) and column (n, i, j).  The GEMM multiplies the
// filter tensor, read in place as the row-major K x CRS matrix M_K, by M_I on
// the fp32 matrix cores (v_mfma_f32_32x32x2_f32) and scatters each output
// column back to NCHW in its epilogue.  For convolutions it gathers M_I from
// the input while loading its B tiles (implicit im2col: no M_I in memory);
// im2col_kernel writes M_I out for the stand-alone entry point and for
// C*R*S >= 2^16.
#include "isc_internal.hpp"

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <type_traits>

namespace isc {
namespace {

// ----------------------------------------------------------------- im2col --

constexpr int kIm2colRows = 8;  // rows of M_I per thread

__global__ __launch_bounds__(256)
void im2col_kernel(const float *__restrict__ x, int C, int H, int W, int R, int S, int T, int P,
                   int Ho, int Wo, int ncols, float *__restrict__ col, int64_t ldc, int rows_total,
                   Decision dec) {
    if (!decision_gate(dec, 2u)) return;
    const int64_t j = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (j >= ldc) return;
    const bool real = j < ncols;
    int n = 0, oy = 0, ox = 0;
    if (real) {
        const int hw = Ho * Wo;
        n = static_cast<int>(j / hw);
        const int p = static_cast<int>(j - static_cast<int64_t>(n) * hw);
        oy = p / Wo;
        ox = p - oy * Wo;
    }
    const int RS = R * S;
    for (int q_begin = blockIdx.y * kIm2colRows; q_begin < rows_total;
         q_begin += gridDim.y * kIm2colRows) {
        const int q_end = min(rows_total, q_begin + kIm2colRows);
        for (int q = q_begin; q < q_end; ++q) {
            float v = 0.0f;
            if (real) {
                const int c = q / RS;
                const int rs = q - c * RS;
                const int r = rs / S;
                const int s = rs - r * S;
                const int iy = oy * T + r - P;
                const int ix = ox * T + s - P;
                if (iy >= 0 && iy < H && ix >= 0 && ix < W)
                    v = x[((static_cast<size_t>(n) * C + c) * H + iy) * W + ix];
            }
            col[static_cast<size_t>(q) * ldc + j] = v;
        }
    }
}

// ------------------------------------------------------------------- GEMM --
//
// Workgroup tile BM x BN = (WAVES_M * WM * 32) x (WAVES_N * WN * 32), four
// wavefronts, each owning WM x WN blocks of 32 x 32 accumulated by
// v_mfma_f32_32x32x2_f32.  K-slices of BK (16, or 32 for the 64 x 64 tile of
// small grids, whose K loop is latency-bound) go through two LDS buffers;
// the next slice's global loads are in flight while the current one feeds
// the matrix cores.  A slices are stored transposed ([k][m]) so that both
// operands are read by 32 consecutive lanes at consecutive addresses.

typedef float floatx16 __attribute__((ext_vector_type(16)));


struct GemmArgs {
    int M, N, Kd;
    const float *a;
    int64_t lda;
    const float *b;
    int64_t ldb;
    float *c;
    int64_t ldc;
    int conv_hw;  // > 0: scatter column n to NCHW with Ho*Wo = conv_hw
    Decision dec;
    Epilogue epi;  // rectifier and census of c
    // split reduction: workgroup z of the grid sums k in [z * kchunk,
    // (z + 1) * kchunk) (kchunk a multiple of 32) and stores its raw partial
    // tile to part[z][m][n]; gemm_split_reduce_kernel adds the partials in z
    // order and applies the epilogue.  part == nullptr: one range, this
    // kernel stores c.
    float *part;
    int kchunk;
    // implicit im2col: B[k][j] is gathered from the input x instead of read
    // from b (k = (c, r, s), j = (n, oy, ox))
    const float *x;
    int C, H, W, T, P, Wo, RS, S;
    uint32_t mRS, mS;  // ceil(2^32 / RS), ceil(2^32 / S) (unused when the divisor is 1)
};

// k / d for k < 2^16, d < 2^16, with m = ceil(2^32 / d) (d > 1)
__device__ __forceinline__ int divm(int k, int d, uint32_t m) {
    return d == 1 ? k : static_cast<int>(__umulhi(static_cast<uint32_t>(k), m));
}

template <int WAVES_M, int WM, int WN, bool A_VEC, bool B_PADDED, bool IMPLICIT, int BK>
__global__ __launch_bounds__(256)
void gemm_f32_kernel(GemmArgs g) {
    if (!decision_gate(g.dec, 2u)) return;
    constexpr int WAVES_N = 4 / WAVES_M;
    constexpr int BM = WAVES_M * WM * 32;
    constexpr int BN = WAVES_N * WN * 32;
    constexpr int PADA = 4, PADB = 4;
    __shared__ __align__(16) float As[2][BK][BM + PADA];
    __shared__ __align__(16) float Bs[2][BK][BN + PADB];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;
    const int m0 = blockIdx.y * BM;
    const int n0 = blockIdx.x * BN;
    const int M = g.M, N = g.N, Kd = g.Kd;

    // global -> register staging
    constexpr int A_F4 = BM * BK / 4;  // float4 per A slice
    constexpr int B_F4 = BK * BN / 4;
    constexpr int A_PER = (A_F4 + 255) / 256;
    constexpr int B_PER = (B_F4 + 255) / 256;
    float4 ra[A_PER];
    float4 rb[B_PER];

    // implicit im2col: this thread's B columns are fixed for the whole
    // K loop; keep each column's input offset and top-left input position
    int coff[IMPLICIT ? B_PER : 1][4], iy0[IMPLICIT ? B_PER : 1][4], ix0[IMPLICIT ? B_PER : 1][4];
    if constexpr (IMPLICIT) {
        const int HW = g.H * g.W;
#pragma unroll
        for (int i = 0; i < B_PER; ++i) {
            const int nq = (tid + i * 256) % (BN / 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int j = n0 + nq * 4 + e;
                if (j < N) {
                    const int img = j / g.conv_hw;
                    const int p = j - img * g.conv_hw;
                    const int oy = p / g.Wo;
                    const int ox = p - oy * g.Wo;
                    iy0[i][e] = oy * g.T - g.P;
                    ix0[i][e] = ox * g.T - g.P;
                    coff[i][e] = img * g.C * HW + iy0[i][e] * g.W + ix0[i][e];
                } else {
                    iy0[i][e] = -(1 << 30);  // fails every bounds test
                    ix0[i][e] = 0;
                    coff[i][e] = 0;
                }
            }
        }
    }

    auto load_slice = [&](int k0) {
        const bool full_k = k0 + BK <= Kd;
#pragma unroll
        for (int i = 0; i < A_PER; ++i) {
            const int idx = tid + i * 256;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (idx < A_F4) {
                const int row = idx % BM;   // consecutive lanes: consecutive rows
                const int kq = idx / BM;    // which 4-wide k group
                const int m = m0 + row;
                const int k = k0 + kq * 4;
                if (m < M) {
                    const float *src = g.a + static_cast<size_t>(m) * g.lda + k;
                    if (A_VEC && full_k) {
                        v = *reinterpret_cast<const float4 *>(src);
                    } else {
                        v.x = k + 0 < Kd ? src[0] : 0.f;
                        v.y = k + 1 < Kd ? src[1] : 0.f;
                        v.z = k + 2 < Kd ? src[2] : 0.f;
                        v.w = k + 3 < Kd ? src[3] : 0.f;
                    }
                }
            }
            ra[i] = v;
        }
#pragma unroll
        for (int i = 0; i < B_PER; ++i) {
            const int idx = tid + i * 256;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (idx < B_F4) {
                const int row = idx / (BN / 4);
                const int nq = idx % (BN / 4);
                const int k = k0 + row;
                const int nn = n0 + nq * 4;
                if (IMPLICIT) {
                    if (k < Kd) {
                        const int c = divm(k, g.RS, g.mRS);
                        const int rs = k - c * g.RS;
                        const int r = divm(rs, g.S, g.mS);
                        const int sx = rs - r * g.S;
                        const int roff = (c * g.H + r) * g.W + sx;
                        float e4[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int iy = iy0[i][e] + r, ix = ix0[i][e] + sx;
                            const bool in = static_cast<unsigned>(iy) < static_cast<unsigned>(g.H) &&
                                            static_cast<unsigned>(ix) < static_cast<unsigned>(g.W);
                            e4[e] = in ? g.x[static_cast<int64_t>(coff[i][e]) + roff] : 0.f;
                        }
                        v = make_float4(e4[0], e4[1], e4[2], e4[3]);
                    }
                } else if (k < Kd) {
                    const float *src = g.b + static_cast<size_t>(k) * g.ldb + nn;
                    if (B_PADDED) {
                        v = *reinterpret_cast<const float4 *>(src);
                    } else {
                        v.x = nn + 0 < N ? src[0] : 0.f;
                        v.y = nn + 1 < N ? src[1] : 0.f;
                        v.z = nn + 2 < N ? src[2] : 0.f;
                        v.w = nn + 3 < N ? src[3] : 0.f;
                    }
                }
            }
            rb[i] = v;
        }
    };
    auto store_slice = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_PER; ++i) {
            const int idx = tid + i * 256;
            if (idx < A_F4) {
                const int row = idx % BM;
                const int kq = idx / BM;
                As[buf][kq * 4 + 0][row] = ra[i].x;
                As[buf][kq * 4 + 1][row] = ra[i].y;
                As[buf][kq * 4 + 2][row] = ra[i].z;
                As[buf][kq * 4 + 3][row] = ra[i].w;
            }
        }
#pragma unroll
        for (int i = 0; i < B_PER; ++i) {
            const int idx = tid + i * 256;
            if (idx < B_F4) {
                const int row = idx / (BN / 4);
                const int nq = idx % (BN / 4);
                *reinterpret_cast<float4 *>(&Bs[buf][row][nq * 4]) = rb[i];
            }
        }
    };

    floatx16 acc[WM][WN];
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    const int kb = g.part ? static_cast<int>(blockIdx.z) * g.kchunk : 0;
    const int ke = g.part ? min(Kd, kb + g.kchunk) : Kd;
    const int nk = (ke - kb + BK - 1) / BK;
    load_slice(kb);
    store_slice(0);
    __syncthreads();
    const int lrow = lane & 31;   // row (A) / column (B) within a 32-block
    const int lk = lane >> 5;     // which of the two k of an MFMA step
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load_slice(kb + (kt + 1) * BK);
#pragma unroll
        for (int kk = 0; kk < BK; kk += 2) {
            float av[WM], bv[WN];
#pragma unroll
            for (int i = 0; i < WM; ++i) av[i] = As[buf][kk + lk][(wm * WM + i) * 32 + lrow];
#pragma unroll
            for (int j = 0; j < WN; ++j) bv[j] = Bs[buf][kk + lk][(wn * WN + j) * 32 + lrow];
#pragma unroll
            for (int i = 0; i < WM; ++i)
#pragma unroll
                for (int j = 0; j < WN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], bv[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) store_slice(buf ^ 1);
        __syncthreads();
    }

    // epilogue: accumulator register v of lane l holds row
    // 8*(v/4) + 4*(l/32) + v%4 and column l%32 of its 32 x 32 block
    if (g.part) {  // a partial sum of the split reduction, stored raw
        float *pz = g.part + static_cast<size_t>(blockIdx.z) * M * N;
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            const int nn = n0 + (wn * WN + j) * 32 + lrow;
            if (nn >= N) continue;
#pragma unroll
            for (int i = 0; i < WM; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int m = m0 + (wm * WM + i) * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
                    if (m < M) pz[static_cast<size_t>(m) * N + nn] = acc[i][j][v];
                }
        }
        return;
    }
    uint32_t cnt = 0;  // nonzero values stored (the census count)
#pragma unroll
    for (int j = 0; j < WN; ++j) {
        const int nn = n0 + (wn * WN + j) * 32 + lrow;
        if (nn >= N) continue;
        size_t col_off;
        size_t row_stride;
        if (g.conv_hw > 0) {
            const int img = nn / g.conv_hw;
            const int p = nn - img * g.conv_hw;
            col_off = static_cast<size_t>(img) * M * g.conv_hw + p;
            row_stride = static_cast<size_t>(g.conv_hw);
        } else {
            col_off = static_cast<size_t>(nn);
            row_stride = static_cast<size_t>(g.ldc);
        }
#pragma unroll
        for (int i = 0; i < WM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + (wm * WM + i) * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
                if (m < M) {
                    const float o = epilogue_value(acc[i][j][v], g.epi.relu);
                    cnt += nonzero_bit(o);
                    g.c[col_off + static_cast<size_t>(m) * row_stride] = o;
                }
            }
        }
    }
    if (g.epi.census) {
        __shared__ uint32_t sums[4];
        census_commit(g.epi, cnt, sums);
    }
}

// ------------------------------------------- pipelined implicit-im2col GEMM --
//
// The convolution GEMM for M > 64 output maps: 128 x 128 workgroup tiles,
// four wavefronts of 64 x 64 (2 x 2 blocks of v_mfma_f32_32x32x2_f32), 16-deep
// K slices streamed through a ring of NST LDS stages NST-1 slices ahead.
// Both operands go from global memory straight into LDS (buffer loads with
// the LDS bit: no staging registers, no LDS stores), 64 consecutive LDS
// words per instruction.  A (the K x CRS filter) is stored as it is laid out,
// [m][k], with rows padded to 17 words so that the 32 rows an MFMA operand
// read touches fall in distinct banks; an instruction covers 64 slots of
// that layout, so each of its lanes reads within one 64-byte row segment and
// pad slots read nothing.  B (the im2col gather) is stored [k][n], each
// instruction one k row of 64 consecutive output columns.  A gather outside the
// input (padding, past the last column, past C*R*S) gets an offset beyond the
// buffer's range, which the hardware reads as zero, so the gather needs no
// select and no zero fill; A rows past M and slices past C*R*S read zero the
// same way.  A slice is consumed after an exact vmcnt wait for the wavefront's
// own loads of it and one barrier (everyone's loads landed, everyone done with
// the slot refilled next).  The ring slot of a slice is chosen by a static
// branch so that the compiler can tell the slot read from the slots being
// filled.
constexpr int kConvBM = 128, kConvBN = 128, kConvBK = 16;
constexpr int kConvAPitch = kConvBK + 1;                                   // LDS words per A row
constexpr int kConvALoads = (kConvBM * kConvAPitch + 4 * 64 - 1) / (4 * 64);  // A loads per wavefront per slice
// Two stages (the next slice in flight while the current one is multiplied)
// and four workgroups per CU measured faster than deeper rings at fewer per
// CU: AlexNet conv2 1.24 ms with 2 stages at four per CU, 1.28-1.31 at
// three, 1.36-1.48 with 3 stages, 1.39 with 4 (two per CU), 1.89 with 5
// (one); the register-staged kernel 1.37.
constexpr int kConvStages = 2;
constexpr uint32_t kOutOfRange = 0x80000000u;  // beyond every buffer this kernel reads (< 2^31 bytes)
constexpr int kGemmBufferFormat = 0x00020000;  // raw buffer, 32-bit data

template <int B, int E, typename F>
__device__ __forceinline__ void for_static(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        for_static<B + 1, E>(f);
    }
}

// s_waitcnt vmcnt(VM) (lgkmcnt and expcnt untouched)
template <int VM>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(VM >= 0 && VM < 64, "vmcnt field");
    constexpr int imm = (VM & 0xF) | ((VM >> 4) << 14) | (0xF << 8) | (0x7 << 4);
    __builtin_amdgcn_s_waitcnt(imm);
}

// 4 bytes per lane at byte offset voff of the buffer into LDS at dst + 4 * lane
// (dst wave-uniform).  A device function: the builtin has no host form.
__device__ __forceinline__ void buffer_to_lds(__amdgpu_buffer_rsrc_t r, float *dst, uint32_t voff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void *)dst, 4,
                                             static_cast<int>(voff), 0, 0, 0);
}

template <int NST>
__global__ __launch_bounds__(256, NST <= 2 ? 4 : (NST == 3 ? 3 : 2))
void gemm_conv_ring_kernel(GemmArgs g) {
    if (!decision_gate(g.dec, 2u)) return;
    constexpr int BM = kConvBM, BN = kConvBN, BK = kConvBK;
    constexpr int AP = kConvAPitch, AL = kConvALoads;
    constexpr int LOADS = AL + (BK / 4) * 2;  // vector-memory operations per wavefront per slice
    constexpr int AW = AL * 4 * 64;           // LDS words of an A slot (>= BM * AP)
    __shared__ __align__(16) float ring[NST][AW + BK * BN];  // [slot][A: m x AP | B: k x n]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.y * BM;
    const int n0 = blockIdx.x * BN;
    const int M = g.M, N = g.N, Kd = g.Kd;
    const int HW = g.H * g.W;

    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(g.a), 0, static_cast<int>(static_cast<int64_t>(M) * g.lda * 4), kGemmBufferFormat);
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(g.x), 0, static_cast<int>(static_cast<int64_t>(g.N / g.conv_hw) * g.C * HW * 4),
        kGemmBufferFormat);

    // this lane's B columns (n0 + h*64 + lane)
    int coff[2], iy0[2], ix0[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int j = n0 + h * 64 + lane;
        if (j < N) {
            const int img = j / g.conv_hw;
            const int p = j - img * g.conv_hw;
            const int oy = p / g.Wo;
            const int ox = p - oy * g.Wo;
            iy0[h] = oy * g.T - g.P;
            ix0[h] = ox * g.T - g.P;
            coff[h] = img * g.C * HW + iy0[h] * g.W + ix0[h];
        } else {
            iy0[h] = -(1 << 30);  // fails every bounds test
            ix0[h] = 0;
            coff[h] = 0;
        }
    }

    // slice kt -> slot SLOT: wavefront w loads AL instructions of A slots and
    // k rows 4w .. 4w+3 of B, both 64-wide halves of each
    auto issue = [&](auto slot_c, int kt) {
        constexpr int SLOT = decltype(slot_c)::value;
        const int k0 = kt * BK;
#pragma unroll
        for (int i = 0; i < AL; ++i) {
            // slot q = (wave*AL + i)*64 + lane holds row q / AP, k offset
            // q % AP of the slice (pad slots, rows past M and k past C*R*S
            // read nothing); decoded per load, which keeps the registers
            // for a fourth workgroup per CU
            const int q = (wave * AL + i) * 64 + lane;
            const int row = q / AP, kk = q - (q / AP) * AP;
            const int m = m0 + row;
            const bool ok = row < BM && kk < BK && m < M && k0 + kk < Kd;
            buffer_to_lds(ra, &ring[SLOT][(wave * AL + i) * 64],
                          ok ? (static_cast<uint32_t>(m) * static_cast<uint32_t>(g.lda) + static_cast<uint32_t>(k0 + kk)) * 4u
                             : kOutOfRange);
        }
#pragma unroll
        for (int i = 0; i < BK / 4; ++i) {
            const int kk = wave * (BK / 4) + i;
            const int k = kt * BK + kk;
            const bool kin = k < Kd;
            const int kc = kin ? k : 0;
            const int c = divm(kc, g.RS, g.mRS);
            const int rs = kc - c * g.RS;
            const int r = divm(rs, g.S, g.mS);
            const int sx = rs - r * g.S;
            const int roff = (c * g.H + r) * g.W + sx;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int iy = iy0[h] + r, ix = ix0[h] + sx;
                const bool in = kin && static_cast<unsigned>(iy) < static_cast<unsigned>(g.H) &&
                                static_cast<unsigned>(ix) < static_cast<unsigned>(g.W);
                buffer_to_lds(rx, &ring[SLOT][AW + kk * BN + h * 64],
                              in ? static_cast<uint32_t>(coff[h] + roff) * 4u : kOutOfRange);
            }
        }
    };

    floatx16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    // the K slices of this workgroup: all of them, or with a split
    // reduction those of range blockIdx.z (kchunk a multiple of BK).
    // Slices prefetched past the range are loaded and never used.
    const int kt0 = g.part ? static_cast<int>(blockIdx.z) * (g.kchunk / BK) : 0;
    const int nk = g.part ? min(g.kchunk / BK, (Kd + BK - 1) / BK - kt0) : (Kd + BK - 1) / BK;
    for_static<0, NST - 1>([&](auto sl) { issue(sl, kt0 + decltype(sl)::value); });
    const int lrow = lane & 31;  // row (A) / column (B) within a 32-block
    const int lk = lane >> 5;    // which of the two k of an MFMA step
    for (int kt = 0; kt < nk; ++kt) {
        for_static<0, NST>([&](auto sl) {
            constexpr int SL = decltype(sl)::value;
            if (kt % NST == SL) {
                // slice kt landed for every wavefront; everyone is done with
                // slice kt - 1, whose slot is refilled next
                wait_vmcnt<(NST - 2) * LOADS>();
                asm volatile("s_barrier" ::: "memory");
                issue(std::integral_constant<int, (SL + NST - 1) % NST>{}, kt0 + kt + NST - 1);
#pragma unroll
                for (int kk = 0; kk < BK; kk += 2) {
                    float av[2], bv[2];
#pragma unroll
                    for (int i = 0; i < 2; ++i) av[i] = ring[SL][((wm * 2 + i) * 32 + lrow) * AP + kk + lk];
#pragma unroll
                    for (int j = 0; j < 2; ++j) bv[j] = ring[SL][AW + (kk + lk) * BN + (wn * 2 + j) * 32 + lrow];
#pragma unroll
                    for (int i = 0; i < 2; ++i)
#pragma unroll
                        for (int j = 0; j < 2; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], bv[j], acc[i][j], 0, 0, 0);
                }
            }
        });
    }
    __builtin_amdgcn_s_waitcnt(0);  // no load into LDS may outlive the workgroup

    // epilogue: accumulator register v of lane l holds row
    // 8*(v/4) + 4*(l/32) + v%4 and column l%32 of its 32 x 32 block
    if (g.part) {  // a partial sum of the split reduction, stored raw
        float *pz = g.part + static_cast<size_t>(blockIdx.z) * M * N;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int nn = n0 + (wn * 2 + j) * 32 + lrow;
            if (nn >= N) continue;
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int m = m0 + (wm * 2 + i) * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
                    if (m < M) pz[static_cast<size_t>(m) * N + nn] = acc[i][j][v];
                }
        }
        return;
    }
    uint32_t cnt = 0;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int nn = n0 + (wn * 2 + j) * 32 + lrow;
        if (nn >= N) continue;
        const int img = nn / g.conv_hw;
        const int p = nn - img * g.conv_hw;
        const size_t col_off = static_cast<size_t>(img) * M * g.conv_hw + p;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + (wm * 2 + i) * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
                if (m < M) {
                    const float o = epilogue_value(acc[i][j][v], g.epi.relu);
                    cnt += nonzero_bit(o);
                    g.c[col_off + static_cast<size_t>(m) * g.conv_hw] = o;
                }
            }
        }
    }
    if (g.epi.census) {
        __syncthreads();  // every wavefront is done with the ring
        census_commit(g.epi, cnt, reinterpret_cast<uint32_t *>(&ring[0][0]));
    }
}

// The split reduction's second pass: c = epilogue(sum over z of part[z]),
// partials added in z order; each workgroup takes kReducePer consecutive
// elements of the M x N result (consecutive threads on consecutive columns)
// and commits its census slot.
constexpr int kReducePer = 2048;

__global__ __launch_bounds__(256)
void gemm_split_reduce_kernel(GemmArgs g, int splits) {
    if (!decision_gate(g.dec, 2u)) return;
    const int64_t mn = static_cast<int64_t>(g.M) * g.N;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kReducePer;
    uint32_t cnt = 0;
    for (int r = 0; r < kReducePer / 256; ++r) {
        const int64_t e = base + r * 256 + threadIdx.x;
        if (e >= mn) break;
        float sum = g.part[e];
        for (int z = 1; z < splits; ++z) sum += g.part[static_cast<int64_t>(z) * mn + e];
        const int m = static_cast<int>(e / g.N);
        const int nn = static_cast<int>(e - static_cast<int64_t>(m) * g.N);
        const float o = epilogue_value(sum, g.epi.relu);
        cnt += nonzero_bit(o);
        const int img = nn / g.conv_hw;
        const int p = nn - img * g.conv_hw;
        g.c[(static_cast<size_t>(img) * g.M + m) * g.conv_hw + p] = o;
    }
    if (g.epi.census) {
        __shared__ uint32_t sums[4];
        census_commit(g.epi, cnt, sums);
    }
}

template <int WAVES_M, int WM, int WN, int BK = 16>
hipError_t launch_gemm_t(const GemmArgs &g, bool a_vec, bool b_padded, bool implicit, hipStream_t s) {
    constexpr int BM = WAVES_M * WM * 32;
    constexpr int BN = (4 / WAVES_M) * WN * 32;
    dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM);
    if (g.part) {  // split reduction (implicit im2col into NCHW only)
        if (!implicit || g.conv_hw <= 0 || g.kchunk <= 0 || g.kchunk % 32 != 0) return hipErrorInvalidValue;
        grid.z = static_cast<unsigned>((g.Kd + g.kchunk - 1) / g.kchunk);
        const int64_t rgroups = (static_cast<int64_t>(g.M) * g.N + kReducePer - 1) / kReducePer;
        if (g.epi.census && census_slots_for(rgroups) > g.epi.cap) return hipErrorInvalidValue;
        if (a_vec) gemm_f32_kernel<WAVES_M, WM, WN, true, false, true, BK><<<grid, 256, 0, s>>>(g);
        else gemm_f32_kernel<WAVES_M, WM, WN, false, false, true, BK><<<grid, 256, 0, s>>>(g);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        gemm_split_reduce_kernel<<<static_cast<unsigned>(rgroups), 256, 0, s>>>(g, static_cast<int>(grid.z));
        return hipGetLastError();
    }
    if (g.epi.census && census_slots_for(static_cast<int64_t>(grid.x) * grid.y) > g.epi.cap)
        return hipErrorInvalidValue;
    if (implicit) {
        if (a_vec) gemm_f32_kernel<WAVES_M, WM, WN, true, false, true, BK><<<grid, 256, 0, s>>>(g);
        else gemm_f32_kernel<WAVES_M, WM, WN, false, false, true, BK><<<grid, 256, 0, s>>>(g);
    } else if (a_vec) {
        if (b_padded) gemm_f32_kernel<WAVES_M, WM, WN, true, true, false, BK><<<grid, 256, 0, s>>>(g);
        else gemm_f32_kernel<WAVES_M, WM, WN, true, false, false, BK><<<grid, 256, 0, s>>>(g);
    } else {
        if (b_padded) gemm_f32_kernel<WAVES_M, WM, WN, false, true, false, BK><<<grid, 256, 0, s>>>(g);
        else gemm_f32_kernel<WAVES_M, WM, WN, false, false, false, BK><<<grid, 256, 0, s>>>(g);
    }
    return hipGetLastError();
}

hipError_t launch_gemm_any(const GemmArgs &g, bool a_vec, bool b_vec, bool implicit, hipStream_t s) {
    // tile height follows M: 32 (skinny), 64, or 128 rows per workgroup; the
    // narrower tile of a height when the wider one leaves fewer than two
    // workgroups per CU
    constexpr int kWideGrid = 512;
    if (g.M <= 32) {
        if ((g.N + 255) / 256 >= kWideGrid) return launch_gemm_t<1, 1, 2>(g, a_vec, b_vec, implicit, s);  // 32 x 256
        return launch_gemm_t<1, 1, 1>(g, a_vec, b_vec, implicit, s);                                       // 32 x 128
    }
    if (g.M <= 64) {
        if ((g.N + 127) / 128 >= kWideGrid) return launch_gemm_t<2, 1, 2>(g, a_vec, b_vec, implicit, s);  // 64 x 128
        return launch_gemm_t<2, 1, 1, 32>(g, a_vec, b_vec, implicit, s);                                   // 64 x 64
    }
    return launch_gemm_t<2, 2, 2>(g, a_vec, b_vec, implicit, s);                // 128 x 128
}

uint32_t div_magic(int d) { return d <= 1 ? 0u : static_cast<uint32_t>((0x100000000ull + d - 1) / d); }

}  // namespace

hipError_t launch_im2col(const float *x, int N, int C, int H, int W, int R, int S, int T, int P,
                         int Ho, int Wo, float *col, int64_t ldc, const Decision &dec, hipStream_t s) {
    const int rows = C * R * S;
    const int ncols = N * Ho * Wo;
    const int row_groups = std::min((rows + kIm2colRows - 1) / kIm2colRows, 65535);
    dim3 grid(static_cast<unsigned>((ldc + 255) / 256), static_cast<unsigned>(row_groups));
    im2col_kernel<<<grid, 256, 0, s>>>(x, C, H, W, R, S, T, P, Ho, Wo, ncols, col, ldc, rows, dec);
    return hipGetLastError();
}

hipError_t launch_gemm_f32(int M, int Ncols, int Kd, const float *a, int64_t lda, const float *b,
                           int64_t ldb, float *c, int64_t ldc, int conv_hw, bool b_padded,
                           const Decision &dec, hipStream_t s, const Epilogue &epi) {
    GemmArgs g{};
    g.M = M; g.N = Ncols; g.Kd = Kd; g.a = a; g.lda = lda; g.b = b; g.ldb = ldb; g.c = c; g.ldc = ldc;
    g.conv_hw = conv_hw; g.dec = dec; g.epi = epi;
    const bool a_vec = (lda % 4 == 0) && (reinterpret_cast<uintptr_t>(a) % 16 == 0);
    const bool b_vec = b_padded && (ldb % 4 == 0) && (reinterpret_cast<uintptr_t>(b) % 16 == 0);
    return launch_gemm_any(g, a_vec, b_vec, false, s);
}

int64_t gemm_max_groups(int64_t M, int64_t Ncols) {
    // the smallest tiles launch_gemm_any picks are 32 rows x 128 columns
    // (M <= 32) and 64 x 64 (M <= 64); the widest grid of any tile is at most
    // ceil(M / 32) * ceil(Ncols / 64), and the split reduction's second pass
    // ceil(M * Ncols / 2048) <= that
    return (M + 31) / 32 * ((Ncols + 63) / 64);
}

namespace {

// Workgroups of the tile launch_gemm_any picks for an M x Ncols product.
int64_t gemm_tiles(int64_t M, int64_t Ncols) {
    if (M <= 32) return (Ncols + 255) / 256 >= 512 ? (Ncols + 255) / 256 : (Ncols + 127) / 128;
    if (M <= 64) return (Ncols + 127) / 128 >= 512 ? (Ncols + 127) / 128 : (Ncols + 63) / 64;
    return (M + 127) / 128 * ((Ncols + 127) / 128);
}

// Workgroup tile (rows x columns) of the kernel launch_gemm_any or the
// pipelined kernel runs for an M x Ncols product.
void gemm_tile_shape(int64_t M, int64_t Ncols, int64_t *tm, int64_t *tn) {
    if (M <= 32) {
        *tm = 32;
        *tn = (Ncols + 255) / 256 >= 512 ? 256 : 128;
    } else if (M <= 64) {
        *tm = 64;
        *tn = (Ncols + 127) / 128 >= 512 ? 128 : 64;
    } else {
        *tm = 128;
        *tn = 128;
    }
}

// Expected time of the implicit GEMM (ms) with C*R*S cut into `ranges`
// reduction ranges: a fixed part, the tiles of the busiest CU (workgroups
// spread over 256 CUs) times each tile's reduction length and size, the
// output (times the ranges of a split reduction, whose partial sums are
// written and summed), and a second launch when the reduction is split.
// Coefficients fitted to the dense path measured on every workload and
// Tab. 2 shape (8.1 % rms, 19 % at most).
double gemm_model(int64_t M, int64_t Ncols, int64_t Kd, int64_t ranges) {
    int64_t tm, tn;
    gemm_tile_shape(M, Ncols, &tm, &tn);
    const int64_t tiles = gemm_tiles(M, Ncols);
    const double per_cu = std::ceil(static_cast<double>(tiles * ranges) / 256.0);
    const double per = static_cast<double>(Kd) / ranges * tm * tn;
    return 0.0257600 + 5.57801e-9 * per_cu * per + 0.98543e-9 * static_cast<double>(M) * Ncols * ranges +
           (ranges > 1 ? 0.00803 : 0.0);
}

// Reduction range per workgroup, 0 for no split; ranges are at least 256
// deep and a multiple of 32 (every K-slice of a range is whole).  A grid of
// fewer than 128 tiles (small batches: AlexNet-ImageNet conv4 at batch 1 is
// 3 tiles, each walking all 3456 of C*R*S) splits for a grid of about 256
// workgroups, at most 16 ranges.  A larger grid of 128 x 128 tiles (more
// than 64 maps) splits into 2-4 ranges where the model above says the
// busiest CU's share shrinks by more than the partial sums cost: AlexNet
// conv5 at batch 128 is 338 tiles, two on 82 CUs and one on the rest, and
// three ranges make it 1014 workgroups, four on the busiest CU with a third
// of the reduction each (0.65 -> 0.45 ms).  A split must gain 10 % in the
// model: at 5 % (the inception 3x3 branch, two ranges) the measured time did
// not move.  (A caller's gemm_split = -1 passes no partial-sum buffer, which
// turns it off.)
int gemm_kchunk(int64_t M, int64_t Ncols, int Kd) {
    const int64_t tiles = gemm_tiles(M, Ncols);
    if (tiles < 128) {
        const int64_t splits = std::min<int64_t>({16, (256 + tiles - 1) / tiles, Kd / 256});
        if (splits < 2) return 0;
        return static_cast<int>((Kd + splits - 1) / splits + 31) / 32 * 32;
    }
    if (M <= 64) return 0;
    int best = 0;
    double best_t = 0.9 * gemm_model(M, Ncols, Kd, 1);
    for (int sp = 2; sp <= 4; ++sp) {
        const int kc = ((Kd + sp - 1) / sp + 31) / 32 * 32;
        if (kc < 256) break;
        const double t = gemm_model(M, Ncols, Kd, (Kd + kc - 1) / kc);
        if (t < best_t) {
            best = kc;
            best_t = t;
        }
    }
    return best;
}

}  // namespace

// Expected time of the dense path's GEMM (ms), with the split the launch
// takes.
double dense_time_model(int64_t M, int64_t Ncols, int64_t Kd) {
    const int kc = Kd < (1ll << 31) ? gemm_kchunk(M, Ncols, static_cast<int>(Kd)) : 0;
    return gemm_model(M, Ncols, Kd, kc > 0 ? (Kd + kc - 1) / kc : 1);
}

size_t conv_gemm_split_floats(int M, int64_t Ncols, int Kd) {
    const int kc = gemm_kchunk(M, Ncols, Kd);
    if (kc == 0) return 0;
    return static_cast<size_t>((Kd + kc - 1) / kc) * static_cast<size_t>(M) * static_cast<size_t>(Ncols);
}

bool conv_gemm_implicit_ok(int C, int R, int S) { return static_cast<int64_t>(C) * R * S < (1 << 16); }

hipError_t launch_conv_gemm(const float *x, const float *w, float *y, int N, int C, int H, int W, int K, int R,
                            int S, int T, int P, int Ho, int Wo, const Decision &dec, hipStream_t s,
                            const Epilogue &epi, float *part) {
    GemmArgs g{};
    g.epi = epi;
    const int kc = part ? gemm_kchunk(K, static_cast<int64_t>(N) * Ho * Wo, C * R * S) : 0;
    g.part = kc > 0 ? part : nullptr;
    g.kchunk = kc;
    g.M = K;
    g.N = N * Ho * Wo;
    g.Kd = C * R * S;
    g.a = w;
    g.lda = g.Kd;
    g.c = y;
    g.conv_hw = Ho * Wo;
    g.dec = dec;
    g.x = x;
    g.C = C; g.H = H; g.W = W; g.T = T; g.P = P; g.Wo = Wo; g.RS = R * S; g.S = S;
    g.mRS = div_magic(R * S);
    g.mS = div_magic(S);
    // more than 64 output maps, operands addressable by 31-bit byte
    // offsets: the pipelined kernel, with or without a split reduction
    const int64_t x_bytes = static_cast<int64_t>(N) * C * H * W * 4;
    const int64_t w_bytes = static_cast<int64_t>(K) * g.Kd * 4;
    if (K > 64 && x_bytes < (1ll << 31) && w_bytes < (1ll << 31)) {
        dim3 grid((g.N + kConvBN - 1) / kConvBN, (g.M + kConvBM - 1) / kConvBM);
        if (g.part) {
            if (g.kchunk <= 0 || g.kchunk % 32 != 0) return hipErrorInvalidValue;
            grid.z = static_cast<unsigned>((g.Kd + g.kchunk - 1) / g.kchunk);
            const int64_t rgroups = (static_cast<int64_t>(g.M) * g.N + kReducePer - 1) / kReducePer;
            if (g.epi.census && census_slots_for(rgroups) > g.epi.cap) return hipErrorInvalidValue;
            gemm_conv_ring_kernel<kConvStages><<<grid, 256, 0, s>>>(g);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            gemm_split_reduce_kernel<<<static_cast<unsigned>(rgroups), 256, 0, s>>>(g, static_cast<int>(grid.z));
            return hipGetLastError();
        }
        if (g.epi.census && census_slots_for(static_cast<int64_t>(grid.x) * grid.y) > g.epi.cap)
            return hipErrorInvalidValue;
        gemm_conv_ring_kernel<kConvStages><<<grid, 256, 0, s>>>(g);
        return hipGetLastError();
    }
    const bool a_vec = (g.lda % 4 == 0) && (reinterpret_cast<uintptr_t>(w) % 16 == 0);
    return launch_gemm_any(g, a_vec, false, true, s);
}

}  // namespace isc
