// gfx950 kernels of the stage forward.
//
// gemv_kernel  : W4A16 matrix-vector product for up to 8 activation rows.  One
//                wave lane owns one weight row of a 64-row tile and streams
//                16-byte chunks (32 INT4 codes) with non-temporal loads; the
//                activation slice sits in LDS as fp16 pairs and is broadcast to
//                all lanes; codes become fp16 with the 0x6400 mask-and-or trick
//                and are consumed by v_dot2_f32_f16 (fp32 accumulation); the
//                group scale multiplies each chunk's partial dot product, so the
//                dequantized weight is exact.  Prologue: RMSNorm of the input
//                row.  Epilogue: plain store, residual add, or SwiGLU.  K is split
//                over workgroups; the last workgroup of a tile (atomic ticket)
//                sums the partials in a fixed order, so results are deterministic.
// attn_kernel  : split-KV decode/verify attention.  Grid = (slot, kv head,
//                split); 16 lanes read one 256-byte cache row, 16 rows per step
//                per workgroup.  Rows j < P are read through the beam table;
//                rows j >= P are this forward's new k/v, rotated and rounded here
//                and written to the cache by their owner.  Mask and causality
//                decide visibility inside an online softmax (exp2 domain);
//                attn_merge_kernel then combines the split partials.
#include "device.h"

#include <climits>

namespace stg {

__device__ __forceinline__ int dest_row(int r, int row_off, int row_map) {
    if (row_map == 0) return row_off + r;
    return 64 * (r >> 5) + (r & 31) + (row_map == 2 ? 32 : 0);   // gate | up interleave
}

// ------------------------------------------------------------------ repack

__global__ void repack_codes_kernel(const uint8_t* __restrict__ q, int n, int k, uint8_t* __restrict__ w_out,
                                    int nchunk, int row_off, int row_map) {
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= (size_t)n * nchunk) return;
    const int r = (int)(idx / nchunk), c = (int)(idx % nchunk);
    const int kb = (k + 1) / 2;
    const int dr = dest_row(r, row_off, row_map);
    const int t = dr >> 6, lane = dr & 63;
    u32x4 o;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        uint32_t wd = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int kk = c * 32 + d * 8 + e;
            uint32_t nib = 8;
            if (kk < k) {
                const uint8_t byte = q[(size_t)r * kb + (kk >> 1)];
                nib = (kk & 1) ? (byte >> 4) : (byte & 15);
            }
            const int sh = (e & 1) ? (16 + 4 * (e >> 1)) : 4 * (e >> 1);
            wd |= nib << sh;
        }
        o[d] = wd;
    }
    *(u32x4*)(w_out + (((size_t)t * nchunk + c) * 64 + lane) * 16) = o;
}

__global__ void repack_scales_kernel(const uint16_t* __restrict__ s, int n, int ng, uint16_t* __restrict__ s_out,
                                     int ngroups, int row_off, int row_map) {
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= (size_t)n * ng) return;
    const int r = (int)(idx / ng), g = (int)(idx % ng);
    const int dr = dest_row(r, row_off, row_map);
    const int t = dr >> 6, lane = dr & 63;
    s_out[((size_t)t * ngroups + g) * 64 + lane] = s[idx];
}

hipError_t launch_repack(const uint8_t* q, const uint16_t* s, int n, int k, int g, uint8_t* w_out, uint16_t* s_out,
                         int ntiles, int nchunk, int ngroups, int row_off, int row_map, hipStream_t st) {
    (void)ntiles;
    const size_t nc = (size_t)n * nchunk;
    repack_codes_kernel<<<dim3((unsigned)((nc + 255) / 256)), dim3(256), 0, st>>>(q, n, k, w_out, nchunk, row_off, row_map);
    const int ng = (k + g - 1) / g;
    const size_t ns = (size_t)n * ng;
    repack_scales_kernel<<<dim3((unsigned)((ns + 255) / 256)), dim3(256), 0, st>>>(s, n, ng, s_out, ngroups, row_off, row_map);
    return hipGetLastError();
}

// ------------------------------------------------------------------ debug dequant

__global__ void dequant_kernel(PackedMat m, int row_off, int row_map, int n_rows, float* __restrict__ out) {
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= (size_t)n_rows * m.nchunk) return;
    const int r = (int)(idx / m.nchunk), c = (int)(idx % m.nchunk);
    const int dr = dest_row(r, row_off, row_map);
    const int t = dr >> 6, lane = dr & 63;
    const u32x4 w = *(const u32x4*)(m.w + (((size_t)t * m.nchunk + c) * 64 + lane) * 16);
    half2_t h[16];
    unpack_chunk(w, h);
    const float sc = f16_to_f32(m.s[((size_t)t * m.ngroups + c / m.gchunks) * 64 + lane]);
#pragma unroll
    for (int p = 0; p < 16; ++p) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int kk = c * 32 + 2 * p + e;
            if (kk < m.k) out[(size_t)r * m.k + kk] = (float)h[p][e] * sc;
        }
    }
}

hipError_t launch_dequant(const PackedMat& m, int row_off, int row_map, int n_rows, float* out, hipStream_t st) {
    const size_t nc = (size_t)n_rows * m.nchunk;
    dequant_kernel<<<dim3((unsigned)((nc + 255) / 256)), dim3(256), 0, st>>>(m, row_off, row_map, n_rows, out);
    return hipGetLastError();
}

// ------------------------------------------------------------------ GEMV

// Inverse RMS of M input rows of length K, fp32, deterministic order.
template <int MT>
__device__ __forceinline__ void rms_fullrow(const GemvArgs& a, int K, float* rs_s, float* bsum) {
    const int tid = threadIdx.x;
    for (int m = 0; m < a.M; ++m) {
        float ss = 0.f;
        for (int k8 = tid; k8 < K / 8; k8 += 256) {
            float v[8];
            const size_t base = (size_t)m * a.in_ld + 8 * k8;
            if (a.in_dt == DT_F32) {
                const float4 p = *(const float4*)((const float*)a.in + base);
                const float4 q = *(const float4*)((const float*)a.in + base + 4);
                v[0] = p.x; v[1] = p.y; v[2] = p.z; v[3] = p.w; v[4] = q.x; v[5] = q.y; v[6] = q.z; v[7] = q.w;
            } else {
                const u32x4 h = *(const u32x4*)((const uint16_t*)a.in + base);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t w = h[e >> 1];
                    v[e] = half_bits_to_f32((uint16_t)((e & 1) ? (w >> 16) : (w & 0xFFFFu)), a.in_dt);
                }
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
        }
        ss = block_sum256(ss, bsum);
        if (tid == 0) rs_s[m] = rsqrtf(ss / (float)K + a.eps);
    }
}

template <int MT, int CPW>
__global__ __launch_bounds__(256) void gemv_kernel(GemvArgs a) {
    constexpr int CPS = 4 * CPW;                 // chunks per workgroup
    constexpr int KLEN = CPS * 32;               // k values per workgroup
    constexpr int NI = (MT * KLEN / 8 + 255) / 256;
    constexpr int NV = (MT * 64 + 255) / 256;
    __shared__ __attribute__((aligned(16))) uint32_t xs[MT][KLEN / 2];
    __shared__ float red[4][MT][64];
    __shared__ float rs_s[MT];
    __shared__ float bsum[256];
    __shared__ int last_s;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int t = blockIdx.x, s = blockIdx.y;
    const PackedMat W = a.W;
    const int M = a.M;
    const int K = W.k;
    const int c0 = s * CPS;
    const int k0 = c0 * 32;

    // ---- weights of this wave: issue every load first (activation-independent)
    const int cw0 = c0 + wave * CPW;
    const u32x4* wbase = (const u32x4*)W.w + ((size_t)t * W.nchunk + cw0) * 64 + lane;
    u32x4 wv[CPW];
    uint16_t sraw[CPW];
#pragma unroll
    for (int u = 0; u < CPW; ++u) wv[u] = __builtin_nontemporal_load(wbase + (size_t)u * 64);
    const uint16_t* sbase = W.s + (size_t)t * W.ngroups * 64 + lane;
#pragma unroll
    for (int u = 0; u < CPW; ++u) sraw[u] = sbase[(size_t)((cw0 + u) / W.gchunks) * 64];

    // ---- prologue: inverse RMS of each input row
    if (a.rms == RMS_FULLROW) {
        rms_fullrow<MT>(a, K, rs_s, bsum);
    } else if (a.rms == RMS_PARTIALS) {
        // wave w reduces rows w, w + 4, ...: lane l adds tiles l, l + 64, ... in order,
        // then lane 0 receives a fixed-order butterfly sum
        for (int m = wave; m < M; m += 4) {
            float ss = 0.f;
            for (int tt = lane; tt < a.ssq_tiles; tt += 64) ss += a.ssq_in[(size_t)m * a.ssq_tiles + tt];
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
            if (lane == 0) rs_s[m] = rsqrtf(ss / (float)K + a.eps);
        }
    }
    __syncthreads();

    // ---- stage the activation slice [k0, k0 + KLEN) as fp16 pairs, 8 k per item
    {
        float v[NI][8];
        float gm[NI][8];
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int it = tid + 256 * i;
            const int m = it / (KLEN / 8);
            const int kk = k0 + 8 * (it % (KLEN / 8));
            const bool ok = (it < M * (KLEN / 8)) && (kk < K);
            const size_t base = ok ? (size_t)m * a.in_ld + kk : 0;
            if (a.in_dt == DT_F32) {
                const float4 p = *(const float4*)((const float*)a.in + base);
                const float4 q = *(const float4*)((const float*)a.in + base + 4);
                v[i][0] = p.x; v[i][1] = p.y; v[i][2] = p.z; v[i][3] = p.w;
                v[i][4] = q.x; v[i][5] = q.y; v[i][6] = q.z; v[i][7] = q.w;
            } else {
                const u32x4 h = *(const u32x4*)((const uint16_t*)a.in + base);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t w = h[e >> 1];
                    v[i][e] = half_bits_to_f32((uint16_t)((e & 1) ? (w >> 16) : (w & 0xFFFFu)), a.in_dt);
                }
            }
            if (a.rms != RMS_NONE) {
                const u32x4 g = *(const u32x4*)(a.gamma + (ok ? kk : 0));
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t w = g[e >> 1];
                    gm[i][e] = half_bits_to_f32((uint16_t)((e & 1) ? (w >> 16) : (w & 0xFFFFu)), a.gamma_dt);
                }
            }
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (!ok) v[i][e] = 0.f;
        }
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int it = tid + 256 * i;
            if (it < M * (KLEN / 8)) {
                const int m = it / (KLEN / 8);
                const int p0 = 4 * (it % (KLEN / 8));
                if (a.rms != RMS_NONE) {
                    const float rs = rs_s[m];
#pragma unroll
                    for (int e = 0; e < 8; ++e) v[i][e] = (v[i][e] * rs) * gm[i][e];
                }
                u32x4 o;
#pragma unroll
                for (int q = 0; q < 4; ++q) o[q] = pack_f16x2(v[i][2 * q], v[i][2 * q + 1]);
                *(u32x4*)&xs[m][p0] = o;
            }
        }
    }
    __syncthreads();

    // ---- dot products (codes exact in fp16, fp32 accumulation, scale per chunk)
    float acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = 0.f;
#pragma unroll
    for (int u = 0; u < CPW; ++u) {
        half2_t wq[16];
        unpack_chunk(wv[u], wq);
        const float sc = f16_to_f32(sraw[u]);
        const int pc = (wave * CPW + u) * 16;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            if (m < M) {
                const u32x4* xv = (const u32x4*)&xs[m][pc];
                float d = 0.f;
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const u32x4 x4 = xv[q4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        // copy the element out first: a bit_cast of a vector-element
                        // lvalue reads element 0 of the vector
                        const uint32_t xe = x4[e];
                        d = __builtin_amdgcn_fdot2(wq[4 * q4 + e], __builtin_bit_cast(half2_t, xe), d, false);
                    }
                }
                acc[m] += sc * d;
            }
        }
    }

    // ---- reduce the four waves (fixed order)
#pragma unroll
    for (int m = 0; m < MT; ++m) red[wave][m][lane] = acc[m];
    __syncthreads();
    float vals[NV];
#pragma unroll
    for (int q = 0; q < NV; ++q) {
        const int idx = tid + 256 * q;
        vals[q] = 0.f;
        if (idx < M * 64) {
            const int m = idx >> 6, r = idx & 63;
            vals[q] = ((red[0][m][r] + red[1][m][r]) + red[2][m][r]) + red[3][m][r];
        }
    }

    // ---- split-K: the last workgroup of the tile sums every split in split order
    if (a.ksplit > 1) {
        const int ldp = W.ntiles * 64;
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q;
            if (idx < M * 64)
                store_coherent(&a.partial[((size_t)s * M + (idx >> 6)) * ldp + t * 64 + (idx & 63)], vals[q]);
        }
        if (!last_arrival(&a.counters[t], (unsigned)a.ksplit, &last_s)) return;
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q;
            if (idx < M * 64) {
                const float* pp = &a.partial[(size_t)(idx >> 6) * ldp + t * 64 + (idx & 63)];
                const size_t stride = (size_t)M * ldp;
                float v = 0.f;
                int ss = 0;
                for (; ss + 8 <= a.ksplit; ss += 8) {
                    float b8[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) b8[e] = load_coherent(pp + (ss + e) * stride);
#pragma unroll
                    for (int e = 0; e < 8; ++e) v += b8[e];
                }
                for (; ss < a.ksplit; ++ss) v += load_coherent(pp + ss * stride);
                vals[q] = v;
            }
        }
    }

    // ---- epilogue
    if (a.epi == EPI_STORE) {
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q;
            if (idx < M * 64) {
                const int m = idx >> 6, n = t * 64 + (idx & 63);
                if (n < W.n) a.out[(size_t)m * a.out_ld + n] = vals[q];
            }
        }
    } else if (a.epi == EPI_RESID) {
        __syncthreads();
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q;
            if (idx < M * 64) {
                const int m = idx >> 6, r = idx & 63;
                const int n = t * 64 + r;
                float xn = 0.f;
                if (n < W.n) {
                    xn = load_val(a.resid, a.resid_dt, (size_t)m * a.resid_ld + n) + vals[q];
                    a.out[(size_t)m * a.out_ld + n] = xn;
                    if (a.out_act) ((uint16_t*)a.out_act)[(size_t)m * a.out_act_ld + n] = to_half_bits(xn, a.out_act_dt);
                }
                red[0][m][r] = xn * xn;
            }
        }
        __syncthreads();
        if (a.ssq_out && tid < M) {
            float ss = 0.f;
            for (int r = 0; r < 64; ++r) ss += red[0][tid][r];
            a.ssq_out[(size_t)tid * W.ntiles + t] = ss;
        }
    } else {  // EPI_SWIGLU: rows 0..31 of the tile are gate rows, 32..63 the matching up rows
        __syncthreads();
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q;
            if (idx < M * 64) red[0][idx >> 6][idx & 63] = vals[q];
        }
        __syncthreads();
        for (int idx = tid; idx < M * 32; idx += 256) {
            const int m = idx >> 5, r = idx & 31;
            const int f = t * 32 + r;
            if (f < a.n_valid) {
                const float gt = red[0][m][r], up = red[0][m][r + 32];
                a.out[(size_t)m * a.out_ld + f] = (gt / (1.0f + expf(-gt))) * up;
            }
        }
    }
}

template <int MT>
hipError_t launch_gemv_m(const GemvArgs& a, int cpw, hipStream_t st) {
    const dim3 grid(a.W.ntiles, a.ksplit), block(256);
    switch (cpw) {
        case 1: gemv_kernel<MT, 1><<<grid, block, 0, st>>>(a); break;
        case 2: gemv_kernel<MT, 2><<<grid, block, 0, st>>>(a); break;
        case 4: gemv_kernel<MT, 4><<<grid, block, 0, st>>>(a); break;
        case 8: gemv_kernel<MT, 8><<<grid, block, 0, st>>>(a); break;
        case 16: gemv_kernel<MT, 16><<<grid, block, 0, st>>>(a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_gemv(const GemvArgs& a, hipStream_t st) {
    if (a.cps % 4) return hipErrorInvalidValue;
    const int cpw = a.cps / 4;
    switch (a.M) {
        case 1: return launch_gemv_m<1>(a, cpw, st);
        case 2: return launch_gemv_m<2>(a, cpw, st);
        case 3: return launch_gemv_m<3>(a, cpw, st);
        case 4: return launch_gemv_m<4>(a, cpw, st);
        case 5: return launch_gemv_m<5>(a, cpw, st);
        case 6: return launch_gemv_m<6>(a, cpw, st);
        case 7: return launch_gemv_m<7>(a, cpw, st);
        case 8: return launch_gemv_m<8>(a, cpw, st);
        default: return hipErrorInvalidValue;
    }
}

// ------------------------------------------------------------------ GEMM (matrix cores)

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// (x & m) | c, written as plain arithmetic (one v_and_or_b32).  Its results feed
// matrix-core operands, so it must stay visible to the compiler: the wait states
// required between a vector write and a matrix-core read of the same register
// are inserted only for instructions the compiler itself emits.
__device__ __forceinline__ uint32_t and_or_u32(uint32_t m, uint32_t x, uint32_t c) { return (x & m) | c; }

// ------------------------------------------------------------------ prepared-operand products
//
// For 2..64 rows the input of every product is written once by the kernel that
// produces it, in the form the matrix cores take: fp16 h with the values at
// positions 2, 3, 6, 7 of every 8 k divided by 16 (they meet codes decoded as
// 1024 + 16u), plus per 32 k the correction 1032 * sum(h at 0, 1, 4, 5) +
// 72 * sum(h at 2, 3, 6, 7) that removes the decode offsets.  An RMSNorm input
// is prepared as h = x * gamma * c with c the row's previous normalization
// scale; the product multiplies its results by rs / c once rs is known
// (RMSNorm(x) W^T = rs ((x * gamma) W^T)).

__device__ __forceinline__ uint16_t bp_code(float h16, int k) { return f32_to_f16((k & 2) ? h16 * 0.0625f : h16); }
__device__ __forceinline__ float bp_corr(float h16, int k) { return ((k & 2) ? 72.0f : 1032.0f) * h16; }

// Sum over the 64 lanes of a wave, identical in every lane.
__device__ __forceinline__ float wave_sum_all(float v) {
    v = sum16(v);
    uint32_t u = __float_as_uint(v);
    const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    u = __float_as_uint(v);
    const auto q = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

// Largest value / smallest integer over the wave, identical in every lane.
__device__ __forceinline__ float wave_max_all(float v) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ int wave_min_all(int v) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) v = min(v, __shfl_xor(v, o, 64));
    return v;
}

// Sum over aligned groups of 32 lanes, identical in every lane of the group.
__device__ __forceinline__ float sum32_lanes(float v) {
    v += dpp_f<0xB1>(v);              // lane ^ 1
    v += dpp_f<0x4E>(v);              // lane ^ 2
    v += dpp_f<0x124>(v);             // row_ror:4
    v += dpp_f<0x128>(v);             // row_ror:8: the 16-lane row
    const uint32_t u = __float_as_uint(v);
    const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Prepared operands are stored in the order the products read them: per group
// of 128 k, per column block cb (16 rows) and product i (k = 32 lg + 8 i + e
// within the group, lg = 0..3), the 64 lanes' 16 bytes (lane 16 lg + row mod
// 16) one after the other, so every operand load is one contiguous kilobyte.
// Corrections are [group][row][4 chunks of 32 k].
__device__ __forceinline__ size_t bp_index(int m, int k) {
    return ((((size_t)(k >> 7) * 16 + (m >> 4) * 4 + ((k >> 3) & 3)) * 64 + ((k >> 5) & 3) * 16 + (m & 15)) << 3) + (k & 7);
}
__device__ __forceinline__ size_t bc_index(int m, int k) { return ((size_t)(k >> 7) * 64 + m) * 4 + ((k >> 5) & 3); }

// One element of a prepared row: lanes 32 c .. 32 c + 31 of a wave hold k = 32 c' + (lane mod 32)
// of one row (valid = k < K); writes the code and, from lane 0 of the 32, the chunk's correction.
__device__ __forceinline__ void bp_put(uint16_t* bp, float* bc, int kp, int m, int k, float h, bool valid) {
    (void)kp;
    const float h16 = valid ? f16_to_f32(f32_to_f16(h)) : 0.f;
    const float cs = sum32_lanes(valid ? bp_corr(h16, k) : 0.f);
    if (valid) bp[bp_index(m, k)] = bp_code(h16, k);
    if (valid && (k & 31) == 0) bc[bc_index(m, k)] = cs;
}

// First q|k|v input of a forward: RMSNorm of the stage input row m, fully
// normalized (c = rs; the product's factor is 1); rs also goes to rs_out for
// the residual product that prepares the next input.  blockIdx.y takes one
// slice of BPREP_SLICE k: every slice adds the whole row's squares in the same
// order (so all get the same rs) and prepares only its own slice.
constexpr int BPREP_SLICE = 1024;
__global__ __launch_bounds__(256) void bprep_kernel(const void* in, int in_dt, int in_ld, const uint16_t* gamma,
                                                    int gamma_dt, int K, float eps, uint16_t* bp, float* bc, int kp,
                                                    float* rs_out) {
    constexpr int NPT = 32;                              // values per thread held in registers: K <= 8192
    constexpr int SPT = BPREP_SLICE / 256;               // slice values per thread
    __shared__ float red[4];
    const int m = blockIdx.x, tid = threadIdx.x, k0 = BPREP_SLICE * blockIdx.y;
    float v[NPT], xs[SPT], gs[SPT];
    size_t off[NPT], offs[SPT];                          // every load issued before any is used (clamped, then dropped)
#pragma unroll
    for (int i = 0; i < NPT; ++i) off[i] = (size_t)m * in_ld + min(tid + 256 * i, K - 1);
#pragma unroll
    for (int i = 0; i < SPT; ++i) offs[i] = (size_t)m * in_ld + min(k0 + tid + 256 * i, K - 1);
    load_vals(in, in_dt, off, v);
    load_vals(in, in_dt, offs, xs);
#pragma unroll
    for (int i = 0; i < SPT; ++i) gs[i] = half_bits_to_f32(gamma[min(k0 + tid + 256 * i, K - 1)], gamma_dt);
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < NPT; ++i) ss += tid + 256 * i < K ? v[i] * v[i] : 0.f;
    ss = wave_sum_all(ss);
    if ((tid & 63) == 0) red[tid >> 6] = ss;
    __syncthreads();
    const float rs = rsqrtf(((red[0] + red[1]) + (red[2] + red[3])) / (float)K + eps);
#pragma unroll
    for (int i = 0; i < SPT; ++i) {
        const int k = k0 + tid + 256 * i;
        if (k0 + 256 * i < K) bp_put(bp, bc, kp, m, k, xs[i] * rs * gs[i], k < K);   // whole 32-lane groups
    }
    if (blockIdx.y == 0 && tid == 0) rs_out[m] = rs;
}

// Inputs of the row factors: the first 32 of this thread's quarter of row m's
// sums of squares (4 threads per row; loads clamped, then dropped past cnt),
// issued early so that they fly with the first group's loads.
struct RowFactorLoads {
    float v[32];
    float cb;
    int cnt;
    const float* src;
};
__device__ __forceinline__ void row_factor_loads(const GemvArgs& a, RowFactorLoads& r) {
    const int tid = threadIdx.x, m = tid >> 2, part = tid & 3;
    r.cb = 1.f;
    r.cnt = 0;
    r.src = a.ssq_in;
    if (a.norm == 1 && m < a.M) {
        r.cb = a.cb_in[m];
        const int per = (a.ssq_tiles + 3) / 4;
        r.src = a.ssq_in + (size_t)m * a.ssq_tiles + part * per;
        r.cnt = max(0, min(per, a.ssq_tiles - part * per));
        if (r.cnt > 0) {
#pragma unroll
            for (int e = 0; e < 32; ++e) r.v[e] = r.src[min(e, r.cnt - 1)];
        }
    }
}

// Factor of every row m < 64 of a product's results into fs (1 unless the
// input is a deferred RMSNorm: then rs / c, rs from the row's sums of squares,
// added by 4 threads per row in index order and combined in a fixed order);
// with write_rs, rs also goes to a.rs_out.  No barrier: fs is read after the
// workgroup's next one.
__device__ __forceinline__ void row_factors_finish(const GemvArgs& a, int K, bool write_rs, const RowFactorLoads& r,
                                                   float* fs) {
    const int tid = threadIdx.x, m = tid >> 2, part = tid & 3;
    float ss = 0.f;
    if (a.norm == 1 && m < a.M) {
#pragma unroll
        for (int e = 0; e < 32; ++e) ss += (e < r.cnt) ? r.v[e] : 0.f;
        for (int tt = 32; tt < r.cnt; tt += 32) {             // more than 128 partials per row
            float v[32];
#pragma unroll
            for (int e = 0; e < 32; ++e) v[e] = r.src[min(tt + e, r.cnt - 1)];
#pragma unroll
            for (int e = 0; e < 32; ++e) ss += (tt + e < r.cnt) ? v[e] : 0.f;
        }
    }
    ss += dpp_f<0xB1>(ss);                                    // lane ^ 1
    ss += dpp_f<0x4E>(ss);                                    // lane ^ 2: the row's 4 parts
    if (part == 0) {
        float f = 1.f;
        if (a.norm == 1 && m < a.M) {
            const float rs = rsqrtf(ss / (float)K + a.eps);
            f = rs / r.cb;
            if (write_rs && a.rs_out) a.rs_out[m] = rs;
        }
        fs[m] = f;
    }
}

// Product of the prepared input with one matrix: a workgroup's 4 waves take
// one 64-row tile and 4 consecutive ranges of a.kg groups of 128 k; blockIdx.y
// is the split of K (fixed per matrix, so results do not depend on M).  A lane
// loads 16 bytes of codes per row block and group (chunk 4 gi + lane / 16 of row
// 16 rt + lane mod 16): dword i of it is the A operand of the group's i-th
// product, whose k are 32 (4 gi + lane / 16) + 8 i + e; the B operand of that
// product is read from the prepared row at the same k.
template <int NCB>
__global__ __launch_bounds__(256, NCB <= 2 ? 2 : 1) void gemm_bp_kernel(GemvArgs a) {
    constexpr int MP = 16 * NCB;
    constexpr int NV = MP * 64 / 256;
    __shared__ float red[4][MP][65];
    __shared__ float fs[64];
    __shared__ float sres[NCB >= 2 ? MP : 1][64], sgam[64], srs[NCB >= 2 ? MP : 1];   // residual-epilogue inputs read at the start
    __shared__ int last_s;
    const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar loop control
    const int l16 = lane & 15, lg = lane >> 4;
    const int t = blockIdx.x, s = blockIdx.y;
    const PackedMat W = a.W;
    const int M = a.M, K = W.k;
    const int g0 = (4 * s + w) * a.kg, g1 = min(W.ngroups, g0 + a.kg);
    const int kc = a.kp / 32;
    uint32_t magic = 0x64006400u;
    asm volatile("" : "+v"(magic));

    auto ldw = [&](int gi, u32x4 (&wv)[4], u32x2 (&sv)[4]) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            wv[rt] = __builtin_nontemporal_load(
                (const u32x4*)(W.w + (((size_t)t * W.nchunk + 4 * gi + lg) * 64 + 16 * rt + l16) * 16));
            sv[rt] = *(const u32x2*)(W.s + ((size_t)t * W.ngroups + gi) * 64 + 16 * rt + 4 * lg);
        }
    };
    // prepared operand and corrections of one group as stored; entries at k >= K
    // (past the end of a ragged last group) are dropped when the group computes,
    // so nothing waits for these loads before then
    auto ldb = [&](int gi, u32x4 (&bv)[NCB][4], float4 (&cv)[NCB]) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            const int m = 16 * cb + l16;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                bv[cb][i] = *(const u32x4*)(a.bp_in + ((((size_t)gi * 16 + cb * 4 + i) * 64 + lane) << 3));
            cv[cb] = *(const float4*)(a.bc_in + ((size_t)gi * 64 + m) * 4);
        }
    };

    f32x4_t acc[4][NCB];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[rt][cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // Two register sets, each the codes, scales, prepared operand and corrections
    // of one group: while one group computes, the next one's loads are in flight.
    // A group's loads are issued together (loads retire from the wait counter in
    // issue order) and unconditionally (the group index is clamped to the wave's
    // last; a repeated group is simply not computed), and nothing reads them
    // before the group computes, so no branch or select sits between a load and
    // its use and the compiler waits for exactly the loads each product needs.
    u32x4 wr[2][4], br[2][NCB][4];
    u32x2 sr[2][4];
    float4 cr[2][NCB];
    // The products of a group are issued k-slice by k-slice (i outer): the 4 NCB
    // accumulators of the tile are independent, so no product waits for the one
    // before it; each accumulator still adds its four slices in order.
    auto compute = [&](int gi, const u32x4 (&wv)[4], const u32x2 (&sv)[4], u32x4 (&bv)[NCB][4], const float4 (&cq)[NCB]) {
        const int kb = 128 * gi;
        float cv[NCB];
        if (kb + 128 <= K) {                             // a whole group (uniform)
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const float4 c4 = cq[cb];
                cv[cb] = (c4.x + c4.y) + (c4.z + c4.w);
            }
        } else {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {            // in place: the set is reloaded after this group
                    const bool in = kb + 32 * lg + 8 * i < K;
#pragma unroll
                    for (int e = 0; e < 4; ++e) bv[cb][i][e] = in ? bv[cb][i][e] : 0u;
                }
                const float4 c4 = cq[cb];
                cv[cb] = ((kb < K ? c4.x : 0.f) + (kb + 32 < K ? c4.y : 0.f)) + ((kb + 64 < K ? c4.z : 0.f) + (kb + 96 < K ? c4.w : 0.f));
            }
        }
        f32x4_t c[4][NCB];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) c[rt][cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            half8_t A[4];
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                const uint32_t x = wv[rt][i], y = x >> 8;
                u32x4 av;
                av[0] = and_or_u32(0x000F000Fu, x, magic);
                av[1] = and_or_u32(0x00F000F0u, x, magic);
                av[2] = and_or_u32(0x000F000Fu, y, magic);
                av[3] = and_or_u32(0x00F000F0u, y, magic);
                A[rt] = __builtin_bit_cast(half8_t, av);
            }
#pragma unroll
            for (int rt = 0; rt < 4; ++rt)
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb)
                    c[rt][cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A[rt], __builtin_bit_cast(half8_t, bv[cb][i]), c[rt][cb], 0, 0, 0);
        }
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            float scl[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t h = sv[rt][j >> 1];
                scl[j] = f16_to_f32((uint16_t)((j & 1) ? (h >> 16) : (h & 0xFFFFu)));
            }
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[rt][cb][j] = __builtin_fmaf(scl[j], c[rt][cb][j] - cv[cb], acc[rt][cb][j]);
        }
    };
    // each tile starts its range at its own group (rotation by the tile index): at
    // any moment the workgroups read different parts of the prepared operand
    const int n = g1 - g0, rot = n > 0 ? t % n : 0;
    auto G = [&](int q) {
        q = min(q, n - 1) + rot;
        return g0 + (q >= n ? q - n : q);
    };
    // With 17 or more rows the residual epilogue's inputs (the tile's residual
    // rows, the next norm's weights and the rows' rs) are read now by every split
    // of the tile, off the last split's tail; the residual is rewritten only by
    // the tile's last split to arrive, after all have started.  (With 16 rows the
    // added start latency outweighs the shorter tail: measured.)
    constexpr bool PRE = NCB >= 2;
    const bool resid_epi = PRE && a.epi == EPI_RESID;
    float pres[NV], prs = 0.f;
    uint16_t pgam_bits = 0;
    if (resid_epi) {
        size_t off[NV];                                  // clamped to a valid element; outside rows are never used
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q, m = min(idx >> 6, M - 1), n = min(t * 64 + (idx & 63), W.n - 1);
            off[q] = (size_t)m * a.resid_ld + n;
        }
        load_vals(a.resid, a.resid_dt, off, pres);
        if (a.bp_out) {                                  // raw now, converted once every load is out
            pgam_bits = a.gamma_next[min(t * 64 + (tid & 63), W.n - 1)];
            prs = a.rs_in[min(tid, M - 1)];
        }
    }
    // factor of each row (rs / c for a deferred RMSNorm input, else 1): its
    // inputs come from the kernel before; they and the epilogue's inputs are
    // issued before the first group's loads, so nothing below waits for those
    RowFactorLoads rfl;
    row_factor_loads(a, rfl);
    __builtin_amdgcn_sched_barrier(0);
    if (n > 0) {
        ldw(G(0), wr[0], sr[0]);
        ldb(G(0), br[0], cr[0]);
    }
    __builtin_amdgcn_sched_barrier(0);
    row_factors_finish(a, K, t == 0 && s == 0, rfl, fs);
    if constexpr (PRE) {
        if (resid_epi) {
#pragma unroll
            for (int q = 0; q < NV; ++q) {
                const int idx = tid + 256 * q;
                sres[idx >> 6][idx & 63] = pres[q];
            }
            if (tid < 64) sgam[tid] = half_bits_to_f32(pgam_bits, a.gamma_next_dt);
            if (tid < MP) srs[tid] = prs;
        }
    }
    if (n > 0) {
        // group q computes from set q & 1 while group q + 1 loads into the other set:
        // whole pairs of groups, then a last single group
        int q = 0;
        for (; q + 2 <= n; q += 2) {
            ldw(G(q + 1), wr[1], sr[1]);
            ldb(G(q + 1), br[1], cr[1]);
            __builtin_amdgcn_sched_barrier(0);           // the loads issue before this group's products
            compute(G(q), wr[0], sr[0], br[0], cr[0]);
            ldw(G(q + 2), wr[0], sr[0]);
            ldb(G(q + 2), br[0], cr[0]);
            __builtin_amdgcn_sched_barrier(0);
            compute(G(q + 1), wr[1], sr[1], br[1], cr[1]);
        }
        if (q < n) {
            ldw(G(q + 1), wr[1], sr[1]);
            ldb(G(q + 1), br[1], cr[1]);
            __builtin_amdgcn_sched_barrier(0);
            compute(G(q), wr[0], sr[0], br[0], cr[0]);
        }
    }
    // ---- the 4 waves' sums of each output (lane: rows 16 rt + 4 lg + j of column 16 cb + l16), in wave order
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int j = 0; j < 4; ++j) red[w][16 * cb + l16][16 * rt + 4 * lg + j] = acc[rt][cb][j];
    __syncthreads();
    float vals[NV];
#pragma unroll
    for (int q = 0; q < NV; ++q) {
        const int idx = tid + 256 * q, m = idx >> 6, r = idx & 63;
        vals[q] = (red[0][m][r] + red[1][m][r]) + (red[2][m][r] + red[3][m][r]);
    }

    // ---- split-K: the last workgroup of the tile sums every split in split order
    if (a.ksplit > 1) {
        const int ldp = W.ntiles * 64;
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q;
            if (idx < M * 64)
                store_coherent(&a.partial[((size_t)s * M + (idx >> 6)) * ldp + t * 64 + (idx & 63)], vals[q]);
        }
        if (!last_arrival(&a.counters[t], (unsigned)a.ksplit, &last_s)) return;
        const size_t stride = (size_t)M * ldp;
#pragma unroll
        for (int q = 0; q < NV; ++q) vals[q] = 0.f;
        for (int s0 = 0; s0 < a.ksplit; s0 += 4) {
            float b4[NV][4];
#pragma unroll
            for (int q = 0; q < NV; ++q) {
                const int idx = tid + 256 * q;
                const float* pp = &a.partial[(size_t)(idx >> 6) * ldp + t * 64 + (idx & 63)];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    b4[q][e] = (idx < M * 64 && s0 + e < a.ksplit) ? load_coherent(pp + (s0 + e) * stride) : 0.f;
            }
#pragma unroll
            for (int q = 0; q < NV; ++q)
#pragma unroll
                for (int e = 0; e < 4; ++e) vals[q] += b4[q][e];
        }
    }

    // ---- epilogue
    if (a.epi == EPI_STORE) {
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q;
            if (idx < M * 64) {
                const int m = idx >> 6, n = t * 64 + (idx & 63);
                if (n < W.n) a.out[(size_t)m * a.out_ld + n] = vals[q] * fs[m];
            }
        }
    } else if (a.epi == EPI_RESID) {
        // the residual rows, the next norm's weights and the rows' rs (read at the
        // start with 17 or more rows), every load issued before any is used
        float xres[NV], egam[NV], ers[NV];
        if constexpr (!PRE) {
            size_t off[NV];
            uint16_t gbits[NV];
#pragma unroll
            for (int q = 0; q < NV; ++q) {
                const int idx = tid + 256 * q, m = min(idx >> 6, M - 1), n = min(t * 64 + (idx & 63), W.n - 1);
                off[q] = (size_t)m * a.resid_ld + n;
                gbits[q] = a.bp_out ? a.gamma_next[n] : (uint16_t)0;
                ers[q] = a.bp_out ? a.rs_in[m] : 0.f;
            }
            load_vals(a.resid, a.resid_dt, off, xres);
#pragma unroll
            for (int q = 0; q < NV; ++q) egam[q] = half_bits_to_f32(gbits[q], a.gamma_next_dt);
        }
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q;
            const int m = idx >> 6, r = idx & 63;                     // one row per wave: whole waves take part
            const int n = t * 64 + r;
            const bool ok = m < M && n < W.n;
            float xn = 0.f;
            if (ok) {
                float xr;
                if constexpr (PRE) xr = sres[m][r];
                else xr = xres[q];
                xn = xr + vals[q] * fs[m];
                a.out[(size_t)m * a.out_ld + n] = xn;
                if (a.out_act) ((uint16_t*)a.out_act)[(size_t)m * a.out_act_ld + n] = to_half_bits(xn, a.out_act_dt);
            }
            // the row's sum of squares over the tile: row m is this wave's 64 lanes
            const float ss = wave_sum_all(xn * xn);
            if (a.ssq_out && m < M && r == 0) a.ssq_out[(size_t)m * W.ntiles + t] = ss;
            if (a.bp_out && m < M) {                                    // the next product's input
                float c, gm;
                if constexpr (PRE) {
                    c = srs[m];
                    gm = sgam[r];
                } else {
                    c = ers[q];
                    gm = egam[q];
                }
                const float h = ok ? xn * gm * c : 0.f;
                bp_put(a.bp_out, a.bc_out, a.kp, m, n, h, ok);
                if (t == 0 && r == 0) a.cb_out[m] = c;
            }
        }
    } else if (a.epi == EPI_TOP1) {
        // per row: the tile's largest value, its smallest index among equal ones,
        // and the sum of exp(v - max) over the tile (row m is one wave's 64 lanes)
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q;
            const int m = idx >> 6, r = idx & 63;
            const int n = t * 64 + r;
            const bool ok = m < M && n < W.n;
            const float v = ok ? vals[q] * fs[m] : -INFINITY;
            if (ok && a.out) a.out[(size_t)m * a.out_ld + n] = v;
            const float mx = wave_max_all(v);
            const int arg = wave_min_all((ok && v == mx) ? n : INT_MAX);
            const float se = wave_sum_all(ok ? expf(v - mx) : 0.f);
            if (m < M && r == 0) a.top1_part[(size_t)m * W.ntiles + t] = make_float4(mx, __int_as_float(arg), se, 0.f);
        }
    } else {  // EPI_SWIGLU: rows 0..31 of the tile are gate rows, 32..63 the matching up rows
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int idx = tid + 256 * q;
            if (idx < M * 64) red[0][idx >> 6][idx & 63] = vals[q] * fs[idx >> 6];
        }
        __syncthreads();
        for (int i0 = 0; i0 < MP * 32; i0 += 256) {                    // whole waves: two rows each
            const int idx = i0 + tid;
            const int m = idx >> 5, r = idx & 31;
            const int f = t * 32 + r;
            const bool ok = m < M && f < a.n_valid;
            float y = 0.f;
            if (ok) {
                const float gt = red[0][m][r], up = red[0][m][r + 32];
                y = (gt / (1.0f + expf(-gt))) * up;
                a.out[(size_t)m * a.out_ld + f] = y;
            }
            if (a.bp_out && m < M) bp_put(a.bp_out, a.bc_out, a.kp, m, f, y, ok);
        }
    }
}

hipError_t launch_gemm_bp(const GemvArgs& a, hipStream_t st) {
    if (a.M < 1 || a.M > 64 || a.W.gchunks != 4 || a.kg < 1 || a.kp % 128) return hipErrorInvalidValue;
    const dim3 grid(a.W.ntiles, a.ksplit), block(256);
    switch ((a.M + 15) / 16) {
        case 1: gemm_bp_kernel<1><<<grid, block, 0, st>>>(a); break;
        case 2: gemm_bp_kernel<2><<<grid, block, 0, st>>>(a); break;
        case 3: gemm_bp_kernel<3><<<grid, block, 0, st>>>(a); break;
        default: gemm_bp_kernel<4><<<grid, block, 0, st>>>(a); break;
    }
    return hipGetLastError();
}

// ------------------------------------------------------------------ prefill product

// Prepared rows of a prompt: row r of `in` goes to row r mod 64 of block r / 64
// (blocks of 64 * kp codes and 2 * kp corrections).  With gamma, the row is
// RMS-normalized first (its squares added in one fixed order by every slice);
// without, it is taken as it is.  One workgroup per (row, slice of 1024 k).
__global__ __launch_bounds__(256) void bprep_rows_kernel(const void* in, int in_dt, int in_ld, const uint16_t* gamma,
                                                         int gamma_dt, int K, float eps, uint16_t* bp, float* bc, int kp) {
    constexpr int SPT = BPREP_SLICE / 256;
    __shared__ float red[4];
    const int r = blockIdx.x, tid = threadIdx.x, k0 = BPREP_SLICE * blockIdx.y;
    uint16_t* bpb = bp + (size_t)(r >> 6) * 64 * kp;
    float* bcb = bc + (size_t)(r >> 6) * 2 * kp;
    float rs = 1.f;
    if (gamma) {
        float ss = 0.f;
        for (int k0b = 0; k0b < K; k0b += 256 * 8) {
            float v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int k = k0b + tid + 256 * i;
                v[i] = load_val(in, in_dt, (size_t)r * in_ld + min(k, K - 1));
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) ss += (k0b + tid + 256 * i < K) ? v[i] * v[i] : 0.f;
        }
        ss = wave_sum_all(ss);
        if ((tid & 63) == 0) red[tid >> 6] = ss;
        __syncthreads();
        rs = rsqrtf(((red[0] + red[1]) + (red[2] + red[3])) / (float)K + eps);
    }
#pragma unroll
    for (int i = 0; i < SPT; ++i) {
        const int k = k0 + tid + 256 * i;
        const int kc = min(k, K - 1);
        const float x = load_val(in, in_dt, (size_t)r * in_ld + kc);
        const float g = gamma ? half_bits_to_f32(gamma[kc], gamma_dt) : 1.f;
        if (k0 + 256 * i < K) bp_put(bpb, bcb, kp, r & 63, k, x * rs * g, k < K);   // whole 32-lane groups
    }
}

hipError_t launch_bprep_rows(const void* in, int in_dt, int in_ld, const uint16_t* gamma, int gamma_dt, int K, float eps,
                             int n, uint16_t* bp, float* bc, int kp, hipStream_t st) {
    if (K < 1 || n < 1 || kp < K || kp % 128) return hipErrorInvalidValue;
    bprep_rows_kernel<<<dim3(n, (K + BPREP_SLICE - 1) / BPREP_SLICE), 256, 0, st>>>(in, in_dt, in_ld, gamma, gamma_dt, K,
                                                                                   eps, bp, bc, kp);
    return hipGetLastError();
}

// Product of a prompt's prepared rows with one matrix.  A workgroup takes four
// 64-row weight tiles (one per wave) and one 64-token block, over all of K.
// Per group of 128 k: the block's 16 operand fragments (16 KB) are copied into
// LDS by direct loads (each wave four of them) and shared by the four waves;
// each wave decodes its tile's codes into the A operands of
// v_mfma_f32_16x16x32_f16 exactly as gemm_bp_kernel does, and adds
// scale * (products - correction) per row and group.  The next group's
// fragments and codes are loaded while a group computes (two LDS buffers, two
// register sets).  Workgroups are numbered so that those sharing a weight tile
// group run on the same XCD one after the other (its L2 keeps the tiles while
// the token blocks sweep past).
template <int DUMMY>
__global__ __launch_bounds__(256, 1) void gemm_pf_kernel(PfArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t sb[2][16][64][8];
    const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, lg = lane >> 4;
    const int total = a.nwt * a.ntb;
    const int per_xcd = (total + 7) / 8;
    const int q = (int)(blockIdx.x & 7) * per_xcd + (int)(blockIdx.x >> 3);
    if (q >= total) return;                                    // whole workgroup: no barrier is reached
    const int wt = q / a.ntb, tb = q % a.ntb;
    const PackedMat W = a.W;
    const int t = 4 * wt + w;
    const bool has = t < W.ntiles;
    const int tt = has ? t : W.ntiles - 1;                     // loads stay in bounds; results are dropped
    const int K = W.k;
    const int ng = (K + 127) / 128;
    const uint16_t* bpb = a.bp + (size_t)tb * a.bp_blk;
    const float* bcb = a.bc + (size_t)tb * a.bc_blk;
    uint32_t magic = 0x64006400u;
    asm volatile("" : "+v"(magic));

    // one group's operand fragments into LDS buffer `buf`: fragment 4 w + u by wave w
    auto stage_b = [&](int g, int buf) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int f = 4 * w + u;
            __builtin_amdgcn_global_load_lds(bpb + (((size_t)g * 16 + f) * 64 + lane) * 8,
                                             (__attribute__((address_space(3))) void*)&sb[buf][f][0][0], 16, 0, 0);
        }
    };
    // codes and scales of the wave's tile, and the corrections of the block's
    // tokens (summed over the group's valid chunks), for group g
    auto ld_w = [&](int g, u32x4 (&wv)[4], u32x2 (&sv)[4], float (&cs)[4]) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            wv[rt] = __builtin_nontemporal_load((const u32x4*)(W.w + (((size_t)tt * W.nchunk + 4 * g + lg) * 64 + 16 * rt + l16) * 16));
            sv[rt] = *(const u32x2*)(W.s + ((size_t)tt * W.ngroups + g) * 64 + 16 * rt + 4 * lg);
        }
        const int kb = 128 * g;
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
            const float4 c4 = *(const float4*)(bcb + ((size_t)g * 64 + 16 * cb + l16) * 4);
            cs[cb] = ((kb < K ? c4.x : 0.f) + (kb + 32 < K ? c4.y : 0.f)) + ((kb + 64 < K ? c4.z : 0.f) + (kb + 96 < K ? c4.w : 0.f));
        }
    };

    f32x4_t acc[4][4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) acc[rt][cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    u32x4 cw[4], nw[4];
    u32x2 cs2[4], ns2[4];
    float cc[4], nc[4];
    stage_b(0, 0);
    ld_w(0, cw, cs2, cc);
    for (int g = 0; g < ng; ++g) {
        const int buf = g & 1;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");       // this wave's copies and loads of group g are done
        __syncthreads();                                        // and every wave's; the other buffer is free
        const bool more = g + 1 < ng;
        if (more) {                                             // group g + 1 loads while group g computes
            stage_b(g + 1, buf ^ 1);
            ld_w(g + 1, nw, ns2, nc);
        }
        const int kb = 128 * g;
        half8_t A[4][4];
        float scl[4][4];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t x = cw[rt][i], y = x >> 8;
                u32x4 av;
                av[0] = and_or_u32(0x000F000Fu, x, magic);
                av[1] = and_or_u32(0x00F000F0u, x, magic);
                av[2] = and_or_u32(0x000F000Fu, y, magic);
                av[3] = and_or_u32(0x00F000F0u, y, magic);
                A[rt][i] = __builtin_bit_cast(half8_t, av);
            }
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const uint32_t h = cs2[rt][jj >> 1];
                scl[rt][jj] = f16_to_f32((uint16_t)((jj & 1) ? (h >> 16) : (h & 0xFFFFu)));
            }
        }
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
            u32x4 B[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                B[i] = *(const u32x4*)&sb[buf][4 * cb + i][lane][0];
                const bool in = kb + 32 * lg + 8 * i < K;          // past the end of a ragged last group: dropped
#pragma unroll
                for (int e = 0; e < 4; ++e) B[i][e] = in ? B[i][e] : 0u;
            }
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                f32x4_t c = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(A[rt][i], __builtin_bit_cast(half8_t, B[i]), c, 0, 0, 0);
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) acc[rt][cb][jj] = __builtin_fmaf(scl[rt][jj], c[jj] - cc[cb], acc[rt][cb][jj]);
            }
        }
        if (more) {
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                cw[rt] = nw[rt];
                cs2[rt] = ns2[rt];
            }
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) cc[cb] = nc[cb];
        }
    }
    if (!has) return;

    // ---- epilogue: lane holds rows 64 t + 16 rt + 4 lg + j of token 64 tb + 16 cb + l16
    if (a.epi == EPI_SWIGLU) {                                 // rows 0..31 of a tile gate, 32..63 the matching up
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                const int tok = 64 * tb + 16 * cb + l16;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int f = 32 * t + 16 * rt + 4 * lg + j;
                    if (tok < a.n && f < a.n_valid) {
                        const float gt = acc[rt][cb][j], up = acc[rt + 2][cb][j];
                        a.out[(size_t)tok * a.out_ld + f] = (gt / (1.0f + expf(-gt))) * up;
                    }
                }
            }
        return;
    }
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
            const int tok = 64 * tb + 16 * cb + l16;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = 64 * t + 16 * rt + 4 * lg + j;
                if (tok >= a.n || row >= W.n) continue;
                float v = acc[rt][cb][j];
                if (a.epi == EPI_RESID) {
                    v += load_val(a.resid, a.resid_dt, (size_t)tok * a.resid_ld + row);
                    if (a.out_act) ((uint16_t*)a.out_act)[(size_t)tok * a.out_act_ld + row] = to_half_bits(v, a.out_act_dt);
                }
                a.out[(size_t)tok * a.out_ld + row] = v;
            }
        }
}

hipError_t launch_gemm_pf(const PfArgs& a, hipStream_t st) {
    if (a.n < 1 || a.W.gchunks != 4 || a.nwt != (a.W.ntiles + 3) / 4 || a.ntb != (a.n + 63) / 64) return hipErrorInvalidValue;
    const int total = a.nwt * a.ntb;
    const unsigned grid = 8u * (unsigned)((total + 7) / 8);
    gemm_pf_kernel<0><<<dim3(grid), dim3(256), 0, st>>>(a);
    return hipGetLastError();
}

hipError_t launch_bprep(const void* in, int in_dt, int in_ld, const uint16_t* gamma, int gamma_dt, int K, float eps,
                        int M, uint16_t* bp, float* bc, int kp, float* rs_out, hipStream_t st) {
    if (K < 1 || K > 32 * 256) return hipErrorInvalidValue;
    bprep_kernel<<<dim3(M, (K + BPREP_SLICE - 1) / BPREP_SLICE), 256, 0, st>>>(in, in_dt, in_ld, gamma, gamma_dt, K, eps,
                                                                              bp, bc, kp, rs_out);
    return hipGetLastError();
}

// ------------------------------------------------------------------ attention

// Rows [j0, j1) of one split are processed in blocks of ABLK keys whose mask
// bytes and table entries are first staged in LDS; each 16-lane key group then
// loads KB cache rows at once before scoring them.
constexpr int ABLK = 256;
constexpr int KB = 4;

template <int D, int RC>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
    constexpr int EPL = D / 16;
    constexpr int HALF = D / 2;
    __shared__ float lo[KGROUPS][RC][D];
    __shared__ float lm[KGROUPS][RC], ll[KGROUPS][RC];
    __shared__ uint8_t smask[ABLK];
    __shared__ int16_t stab[ABLK];

    const int item = blockIdx.x, g = blockIdx.y, split = blockIdx.z;
    const ItemDev it = a.meta.items[item];
    const ReqDev rq = it.rq;
    const int b = it.slot;
    const int P = rq.P, n = rq.n;
    const int L = P + n;
    int split_len = max(ATTN_MIN_SPLIT, (L + rq.splits - 1) / rq.splits);
    split_len = (split_len + KGROUPS - 1) / KGROUPS * KGROUPS;
    const int nsplit = (L + split_len - 1) / split_len;
    if (split >= nsplit) return;
    const int j0 = split * split_len, j1 = min(L, j0 + split_len);

    const int tid = threadIdx.x, kg = tid >> 4, li = tid & 15;
    const int Hq = a.Hq, Hkv = a.Hkv;
    const int gs = Hq / Hkv;
    const int R = gs * n;
    const size_t lstride = (size_t)rq.S * Hkv * rq.cap * D;
    uint16_t* kl = rq.kc + (size_t)a.layer * lstride;
    uint16_t* vl = rq.vc + (size_t)a.layer * lstride;
    const uint8_t* mask = a.meta.masks + rq.mask_off + (size_t)b * rq.mask_len;
    // per-query-row masks of the slot, [n][mask_len], when the request has them
    const uint8_t* rmask = rq.rowmask_off >= 0 ? a.meta.masks + rq.rowmask_off + (size_t)b * n * rq.mask_len : nullptr;
    const int16_t* tab = rq.table + (size_t)b * rq.cap;
    const int rowbase = rq.row0 + b * n;
    const int d0 = li * EPL;
    const int jc1 = min(j1, P);            // cached rows end here; [max(j0, P), j1) are new rows

    for (int r0 = 0; r0 < R; r0 += RC) {
        float q[RC][EPL];
        int qi[RC];
#pragma unroll
        for (int rr = 0; rr < RC; ++rr) {
            const int r = r0 + rr;
            qi[rr] = -1;
#pragma unroll
            for (int e = 0; e < EPL; ++e) q[rr][e] = 0.f;
            if (r < R) {
                const int i = r / gs, h = g * gs + (r % gs);
                const int m = rowbase + i;
                const int pos = a.meta.positions[m];
                const float* qrow = a.qkv + (size_t)m * a.qkv_ld + (size_t)h * D;
                qi[rr] = i;
#pragma unroll
                for (int e = 0; e < EPL; ++e) {
                    const int d = d0 + e;
                    const bool lo_half = d < HALF;
                    const float x = qrow[d];
                    const float xp = lo_half ? qrow[d + HALF] : qrow[d - HALF];
                    const float2 cs = a.rope[(size_t)pos * HALF + (lo_half ? d : d - HALF)];
                    const float y = lo_half ? (x * cs.x - xp * cs.y) : (x * cs.x + xp * cs.y);
                    q[rr][e] = y * a.qscale;
                }
            }
        }
        float mx[RC], sl[RC], o[RC][EPL];
#pragma unroll
        for (int rr = 0; rr < RC; ++rr) {
            mx[rr] = -INFINITY;
            sl[rr] = 0.f;
#pragma unroll
            for (int e = 0; e < EPL; ++e) o[rr][e] = 0.f;
        }

        auto consume = [&](int j, const float* kf, const float* vf) {
#pragma unroll
            for (int rr = 0; rr < RC; ++rr) {
                if (qi[rr] < 0) continue;
                float sd = 0.f;
#pragma unroll
                for (int e = 0; e < EPL; ++e) sd += q[rr][e] * kf[e];
                sd = sum16(sd);
                if (j > P + qi[rr]) continue;                 // causal over the physical index
                if (rmask && rmask[(size_t)qi[rr] * rq.mask_len + j] == 0) continue;   // hidden from this row
                const float mn = fmaxf(mx[rr], sd);
                const float corr = exp2f(mx[rr] - mn);
                const float p = exp2f(sd - mn);
                sl[rr] = sl[rr] * corr + p;
#pragma unroll
                for (int e = 0; e < EPL; ++e) o[rr][e] = o[rr][e] * corr + p * vf[e];
                mx[rr] = mn;
            }
        };

        // ---- cached rows: read through the beam table
        for (int jb = j0; jb < jc1; jb += ABLK) {
            const int nb = min(ABLK, jc1 - jb);
            __syncthreads();
            for (int x = tid; x < nb; x += 256) {
                smask[x] = mask[jb + x];
                stab[x] = tab[jb + x];
            }
            __syncthreads();
            for (int x0 = kg; x0 < nb; x0 += KGROUPS * KB) {
                uint16_t kb[KB][EPL], vb[KB][EPL];
                bool vis[KB];
#pragma unroll
                for (int u = 0; u < KB; ++u) {
                    const int x = x0 + u * KGROUPS;
                    vis[u] = (x < nb) && smask[x] != 0;      // hidden from every query of the slot
                    if (vis[u]) {
                        const int j = jb + x;
                        const size_t off = (((size_t)stab[x] * Hkv + g) * rq.cap + j) * D + d0;
                        if constexpr (EPL == 8) {
                            *(u32x4*)kb[u] = *(const u32x4*)(kl + off);
                            *(u32x4*)vb[u] = *(const u32x4*)(vl + off);
                        } else {
                            *(u32x2*)kb[u] = *(const u32x2*)(kl + off);
                            *(u32x2*)vb[u] = *(const u32x2*)(vl + off);
                        }
                    }
                }
#pragma unroll
                for (int u = 0; u < KB; ++u) {
                    if (!vis[u]) continue;
                    float kf[EPL], vf[EPL];
#pragma unroll
                    for (int e = 0; e < EPL; ++e) {
                        kf[e] = half_bits_to_f32(kb[u][e], a.kv_dt);
                        vf[e] = half_bits_to_f32(vb[u][e], a.kv_dt);
                    }
                    consume(jb + x0 + u * KGROUPS, kf, vf);
                }
            }
        }

        // ---- this forward's rows: rotate k, round k and v to the cache dtype, append
        for (int j = max(j0, P) + kg; j < j1; j += KGROUPS) {
            if (mask[j] == 0) continue;
            const int i = j - P;
            const int m = rowbase + i;
            const int pos = a.meta.positions[m];
            const float* krow = a.qkv + (size_t)m * a.qkv_ld + (size_t)(Hq + g) * D;
            const float* vrow = a.qkv + (size_t)m * a.qkv_ld + (size_t)(Hq + Hkv + g) * D;
            uint16_t kb[EPL], vb[EPL];
            float kf[EPL], vf[EPL];
#pragma unroll
            for (int e = 0; e < EPL; ++e) {
                const int d = d0 + e;
                const bool lo_half = d < HALF;
                const float x = krow[d];
                const float xp = lo_half ? krow[d + HALF] : krow[d - HALF];
                const float2 cs = a.rope[(size_t)pos * HALF + (lo_half ? d : d - HALF)];
                const float y = lo_half ? (x * cs.x - xp * cs.y) : (x * cs.x + xp * cs.y);
                kb[e] = to_half_bits(y, a.kv_dt);
                vb[e] = to_half_bits(vrow[d], a.kv_dt);
                kf[e] = half_bits_to_f32(kb[e], a.kv_dt);
                vf[e] = half_bits_to_f32(vb[e], a.kv_dt);
            }
            consume(j, kf, vf);
        }
        if (r0 == 0 && !a.no_append) {                          // append: owner of row j writes it
            for (int j = max(j0, P) + kg; j < j1; j += KGROUPS) {
                const int i = j - P;
                const int m = rowbase + i;
                const int pos = a.meta.positions[m];
                const float* krow = a.qkv + (size_t)m * a.qkv_ld + (size_t)(Hq + g) * D;
                const float* vrow = a.qkv + (size_t)m * a.qkv_ld + (size_t)(Hq + Hkv + g) * D;
                const size_t off = (((size_t)b * Hkv + g) * rq.cap + j) * D + d0;
#pragma unroll
                for (int e = 0; e < EPL; ++e) {
                    const int d = d0 + e;
                    const bool lo_half = d < HALF;
                    const float x = krow[d];
                    const float xp = lo_half ? krow[d + HALF] : krow[d - HALF];
                    const float2 cs = a.rope[(size_t)pos * HALF + (lo_half ? d : d - HALF)];
                    const float y = lo_half ? (x * cs.x - xp * cs.y) : (x * cs.x + xp * cs.y);
                    kl[off + e] = to_half_bits(y, a.kv_dt);
                    vl[off + e] = to_half_bits(vrow[d], a.kv_dt);
                }
                if (a.layer == 0 && g == 0 && li == 0) rq.table[(size_t)b * rq.cap + j] = (int16_t)b;
            }
        }

        // ---- merge the 16 key groups (fixed order) into this split's partial
#pragma unroll
        for (int rr = 0; rr < RC; ++rr) {
            if (li == 0) {
                lm[kg][rr] = mx[rr];
                ll[kg][rr] = sl[rr];
            }
#pragma unroll
            for (int e = 0; e < EPL; ++e) lo[kg][rr][d0 + e] = o[rr][e];
        }
        __syncthreads();
        for (int idx = tid; idx < RC * D; idx += 256) {
            const int rr = idx / D, d = idx % D;
            const int r = r0 + rr;
            if (r >= R) continue;
            float M = -INFINITY;
            for (int k2 = 0; k2 < KGROUPS; ++k2) M = fmaxf(M, lm[k2][rr]);
            float O = 0.f, S = 0.f;
            for (int k2 = 0; k2 < KGROUPS; ++k2) {
                const float mk = lm[k2][rr];
                const float w = (mk == -INFINITY) ? 0.f : exp2f(mk - M);
                O += lo[k2][rr][d] * w;
                S += ll[k2][rr] * w;
            }
            const int i = r / gs, h = g * gs + (r % gs);
            const int m = rowbase + i;
            float* pp = a.part + (((size_t)m * Hq + h) * a.nsplit_max + split) * (D + 2);
            store_coherent(pp + 2 + d, O);
            if (d == 0) {
                store_coherent(pp, M);
                store_coherent(pp + 1, S);
            }
        }
        __syncthreads();
    }
}

// Merge of the split partials: one workgroup per (activation row, query head),
// one thread per output element; splits combined in split order.
template <int D>
__global__ __launch_bounds__(D) void attn_merge_kernel(AttnArgs a) {
    __shared__ float wgt[ATTN_MAX_SPLITS];
    __shared__ float inv_s;
    const int m = blockIdx.x, h = blockIdx.y, d = threadIdx.x;
    const ReqDev rq = a.meta.items[a.meta.row_item[m]].rq;    // the request of row m
    const int L = rq.P + rq.n;
    int split_len = max(ATTN_MIN_SPLIT, (L + rq.splits - 1) / rq.splits);
    split_len = (split_len + KGROUPS - 1) / KGROUPS * KGROUPS;
    const int nsplit = (L + split_len - 1) / split_len;
    const float* pp = a.part + ((size_t)m * a.Hq + h) * a.nsplit_max * (D + 2);
    if (d < 32) {
        float M = -INFINITY;
        for (int s2 = d; s2 < nsplit; s2 += 32) M = fmaxf(M, pp[(size_t)s2 * (D + 2)]);
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o, 32));
        float S = 0.f;
        for (int s2 = d; s2 < nsplit; s2 += 32) {
            const float ms = pp[(size_t)s2 * (D + 2)];
            const float w = (ms == -INFINITY) ? 0.f : exp2f(ms - M);
            wgt[s2] = w;
            S += pp[(size_t)s2 * (D + 2) + 1] * w;
        }
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) S += __shfl_xor(S, o, 32);
        if (d == 0) inv_s = 1.0f / S;
    }
    __syncthreads();
    float O = 0.f;
    for (int s2 = 0; s2 < nsplit; ++s2) O += pp[(size_t)s2 * (D + 2) + 2 + d] * wgt[s2];
    a.out[(size_t)m * a.out_ld + (size_t)h * D + d] = O * inv_s;
    if (a.bp_out)                                            // the o product's input (64-row blocks)
        bp_put(a.bp_out + (size_t)(m >> 6) * 64 * a.kp, a.bc_out + (size_t)(m >> 6) * 2 * a.kp, a.kp, m & 63, h * D + d,
               O * inv_s, true);
}

// ------------------------------------------------------------------ matrix-core attention
//
// Same work split, partial format and append as attn_kernel, with the products
// on the matrix cores: every query vector of the (item, kv head) meets each
// 32-key step once.  Per 16-key subtile the scores are S^T = K Q^T (cache rows
// are the A operand as stored; q is split into a rounded part and its residual,
// both in the cache dtype, so the scores carry nearly fp32 precision), and the
// output is O^T += V^T P^T with P^T taken straight from the score registers
// (lane l holds keys 4 (l / 16) + j of both subtiles: exactly the k-slots of
// the B operand) and V^T read from a transposed copy of the value tile in LDS
// whose key slots follow the same order.  Keys a query may not see enter as
// zero rows with a -inf score.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
constexpr int AK = 32;                   // keys per step
constexpr int ACH = 512;                 // keys whose table entry and mask byte are staged at once

template <int KVDT>
__device__ __forceinline__ f32x4_t mma_kv(const u32x4& A, const u32x4& B, f32x4_t c) {
    if constexpr (KVDT == DT_BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, A), __builtin_bit_cast(bf16x8_t, B), c,
                                                       0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, A), __builtin_bit_cast(half8_t, B), c, 0,
                                                      0, 0);
}
template <int KVDT>
__device__ __forceinline__ uint16_t kv_round(float f) { return KVDT == DT_BF16 ? f32_to_bf16(f) : f32_to_f16(f); }
template <int KVDT>
__device__ __forceinline__ float kv_float(uint16_t b) { return KVDT == DT_BF16 ? bf16_to_f32(b) : f16_to_f32(b); }
// Two floats rounded to the cache dtype (to nearest even) and packed, low half
// first: one v_cvt_pk_bf16_f32 for bf16.  Equal to kv_round of each for every
// finite input that is not an fp32 denormal (the probabilities it packs never are).
template <int KVDT>
__device__ __forceinline__ uint32_t kv_pack2(float lo, float hi) {
    if constexpr (KVDT == DT_BF16) {
        typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
        const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
        return __builtin_bit_cast(uint32_t, v);
    } else {
        return (uint32_t)kv_round<KVDT>(lo) | ((uint32_t)kv_round<KVDT>(hi) << 16);
    }
}

// The values of v in this lane and in lane ^ sh (sh = 16 or 32): every lane of
// the pair receives the lower lane's value in a and the upper lane's in b.
__device__ __forceinline__ void lane_pair_k(float v, int sh, float& a, float& b) {
    const uint32_t u = __float_as_uint(v);
    if (sh == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
        a = __uint_as_float(r[0]);
        b = __uint_as_float(r[1]);
    } else {
        const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
        a = __uint_as_float(r[0]);
        b = __uint_as_float(r[1]);
    }
}

// QTW: query tiles per wave per pass (which wave computes a query vector, and
// when, does not change its arithmetic).
template <int D, int KVDT, int QTW, bool REC = false>
__global__ __launch_bounds__(256, QTW == 1 ? 2 : 1) void attn_mma_kernel(AttnArgs a) {
    constexpr int HALF = D / 2;
    constexpr int NCH = D / 8;               // 16-byte chunks per cache row
    constexpr int DB = D / 32;               // k-blocks of the score products
    constexpr int MB = D / 16;               // row blocks of O^T
    constexpr int NU = AK * NCH / 256;       // chunks per thread per step (K and V each)
    constexpr int NS = ACH / 256;            // staged table entries per thread
    constexpr int VST = 40;                  // V^T row stride in elements (32 key slots + padding)
    static_assert(NU >= 1 && AK * NCH % 256 == 0, "tile staging");
    __shared__ __attribute__((aligned(16))) uint16_t ks[2][AK][D];   // key rows, chunk c at c ^ (key mod NCH)
    __shared__ __attribute__((aligned(16))) uint16_t vt[2][D][VST];  // values transposed, key slots permuted
    __shared__ int16_t stab[ACH];                                    // physical slot of each key of the chunk
    __shared__ __attribute__((aligned(16))) uint8_t smk[ACH];        // its mask byte (read as words)

    const int item = blockIdx.x, g = blockIdx.y, split = blockIdx.z;
    const ItemDev it = a.meta.items[item];
    const ReqDev rq = it.rq;
    const int b = it.slot;
    const int P = rq.P, n = rq.n;
    const int L = P + n;
    int split_len = max(ATTN_MIN_SPLIT, (L + rq.splits - 1) / rq.splits);
    split_len = (split_len + KGROUPS - 1) / KGROUPS * KGROUPS;
    const int nsplit = (L + split_len - 1) / split_len;
    if (split >= nsplit) return;
    const int j0 = split * split_len, j1 = min(L, j0 + split_len);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int ql = lane & 15, lg = lane >> 4;
    const int Hq = a.Hq, Hkv = a.Hkv;
    const int gs = Hq / Hkv;
    const int R = gs * n;
    const int nqt = (R + 15) / 16;
    const size_t lstride = (size_t)rq.S * Hkv * rq.cap * D;
    uint16_t* kl = rq.kc + (size_t)a.layer * lstride;
    uint16_t* vl = rq.vc + (size_t)a.layer * lstride;
    const uint8_t* mask = a.meta.masks + rq.mask_off + (size_t)b * rq.mask_len;
    // per-query-row masks of the slot, [n][mask_len], when the request has them
    const uint8_t* rmask = rq.rowmask_off >= 0 ? a.meta.masks + rq.rowmask_off + (size_t)b * n * rq.mask_len : nullptr;
    const int16_t* tab = rq.table + (size_t)b * rq.cap;
    const int rowbase = rq.row0 + b * n;

    // ---- one step's keys (chunk-relative key x0 + k): cache rows through the
    // table, this forward's rows from q|k|v.  Cache rows are loaded without
    // branches (clamped to an allocated row; whether a chunk is kept is a bit
    // applied when it is staged), so the mask and table reads are all in flight
    // at once and nothing waits for the loads before the staging.
    u32x4 kreg[NU], vreg[NU];
    uint32_t keep = 0u;
    int c0 = j0, c1 = j0;                                    // keys of the staged chunk
    auto fetch = [&](int x0, bool append) {
        uint32_t kb_ = 0u;
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int q = tid + 256 * u, k = q / NCH, c = q % NCH;
            const int x = min(x0 + k, ACH - 1), j = c0 + x0 + k;
            const bool cached = j < min(c1, P);
            const int slot = cached ? (int)stab[x] : b;
            const size_t off = (((size_t)slot * Hkv + g) * rq.cap + (cached ? j : 0)) * D + 8 * c;
            kreg[u] = *(const u32x4*)(kl + off);
            vreg[u] = *(const u32x4*)(vl + off);
            kb_ |= ((cached && smk[x] != 0) ? 1u : 0u) << u;
        }
        if (c0 + x0 + AK > P && c0 + x0 < c1) {              // the step holds rows of this forward (uniform)
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int q = tid + 256 * u, k = q / NCH, c = q % NCH;
                const int x = min(x0 + k, ACH - 1), j = c0 + x0 + k;
                if (j < P || j >= c1) continue;
                const int i = j - P;
                const int m = rowbase + i;
                const int pos = a.meta.positions[m];
                const float* krow = a.qkv + (size_t)m * a.qkv_ld + (size_t)(Hq + g) * D;
                const float* vrow = a.qkv + (size_t)m * a.qkv_ld + (size_t)(Hq + Hkv + g) * D;
                uint16_t kb[8], vb[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int d = 8 * c + e;
                    const bool lo_half = d < HALF;
                    const float xk = krow[d];
                    const float xp = lo_half ? krow[d + HALF] : krow[d - HALF];
                    const float2 cs = a.rope[(size_t)pos * HALF + (lo_half ? d : d - HALF)];
                    const float y = lo_half ? (xk * cs.x - xp * cs.y) : (xk * cs.x + xp * cs.y);
                    kb[e] = kv_round<KVDT>(y);
                    vb[e] = kv_round<KVDT>(vrow[d]);
                }
                u32x4 kk, vv;
#pragma unroll
                for (int w2 = 0; w2 < 4; ++w2) {
                    kk[w2] = (uint32_t)kb[2 * w2] | ((uint32_t)kb[2 * w2 + 1] << 16);
                    vv[w2] = (uint32_t)vb[2 * w2] | ((uint32_t)vb[2 * w2 + 1] << 16);
                }
                if (append) {                                // append: owner of row j writes it
                    const size_t off = (((size_t)b * Hkv + g) * rq.cap + j) * D + 8 * c;
                    *(u32x4*)(kl + off) = kk;
                    *(u32x4*)(vl + off) = vv;
                    if (a.layer == 0 && g == 0 && c == 0) rq.table[(size_t)b * rq.cap + j] = (int16_t)b;
                }
                kreg[u] = kk;
                vreg[u] = vv;
                kb_ |= (smk[x] != 0 ? 1u : 0u) << u;
            }
        }
        keep = kb_;
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int q = tid + 256 * u, k = q / NCH, c = q % NCH;
            const bool kp_ = (keep >> u) & 1u;               // dropped chunks enter as zero rows
            const u32x4 kv = kreg[u], vv = vreg[u];
            *(u32x4*)&ks[buf][k][8 * (c ^ (k % NCH))] = u32x4{kp_ ? kv[0] : 0u, kp_ ? kv[1] : 0u, kp_ ? kv[2] : 0u, kp_ ? kv[3] : 0u};
            const int slot = 8 * ((k & 15) >> 2) + 4 * (k >> 4) + (k & 3);
#pragma unroll
            for (int e = 0; e < 8; ++e) vt[buf][8 * c + e][slot] = kp_ ? (uint16_t)(vv[e >> 1] >> (16 * (e & 1))) : (uint16_t)0;
        }
    };

    // table entries and mask bytes of the first chunk
    int16_t ptab[NS];
    uint8_t pmsk[NS];
#pragma unroll
    for (int t2 = 0; t2 < NS; ++t2) {
        const int j = j0 + tid + 256 * t2;
        const bool in = j < min(j1, j0 + ACH);
        pmsk[t2] = in ? mask[j] : 0;
        ptab[t2] = (in && j < P) ? tab[j] : (int16_t)b;
    }
    // ---- the first chunk's mask bytes and table entries are staged and its first
    // step's loads issued before the queries are set up: they fly during it
    c1 = min(j1, j0 + ACH);
#pragma unroll
    for (int t2 = 0; t2 < NS; ++t2) {
        smk[tid + 256 * t2] = pmsk[t2];
        stab[tid + 256 * t2] = ptab[t2];
    }
    __syncthreads();
    fetch(0, !a.no_append);
    for (int qg = 0; qg < nqt; qg += 4 * QTW) {
        // ---- this wave's query tiles: rotated, scaled, split into rounded part and residual
        u32x4 qh[QTW][DB], qr[QTW][DB];
        int qtok[QTW];
        float mrun[QTW], lsum[QTW];
        f32x4_t o[QTW][MB];
#pragma unroll
        for (int u = 0; u < QTW; ++u) {
            const int qt = qg + wave + 4 * u;
            const int r = 16 * qt + ql;
            const bool ok = qt < nqt && r < R;
            const int i = ok ? r / gs : 0, h = g * gs + (ok ? r % gs : 0);
            const int m = rowbase + i;
            const float* qrow = a.qkv + (size_t)m * a.qkv_ld + (size_t)h * D;
            qtok[u] = ok ? i : n;
            // every load of the tile at once (row 0 of the item stands in for a missing
            // row): q and its rotary partners, then (cos, sin) at the row's position
            float4 qa[DB][2], qp[DB][2], rc[DB][4];
#pragma unroll
            for (int ib = 0; ib < DB; ++ib) {
                const int d0 = 32 * ib + 8 * lg;
                const bool lo_half = d0 < HALF;
#pragma unroll
                for (int h2 = 0; h2 < 2; ++h2) {
                    qa[ib][h2] = ((const float4*)(qrow + d0))[h2];
                    qp[ib][h2] = ((const float4*)(qrow + (lo_half ? d0 + HALF : d0 - HALF)))[h2];
                }
            }
            const int pos = a.meta.positions[m];
#pragma unroll
            for (int ib = 0; ib < DB; ++ib) {
                const int d0 = 32 * ib + 8 * lg;
                const float4* r4 = (const float4*)(a.rope + (size_t)pos * HALF + (d0 < HALF ? d0 : d0 - HALF));
#pragma unroll
                for (int h4 = 0; h4 < 4; ++h4) rc[ib][h4] = r4[h4];
            }
#pragma unroll
            for (int ib = 0; ib < DB; ++ib) {
                // dims d0 .. d0 + 7 lie in one rotary half
                const int d0 = 32 * ib + 8 * lg;
                const bool lo_half = d0 < HALF;
                float xv[8], xpv[8], cv[8], sv[8];
#pragma unroll
                for (int h2 = 0; h2 < 2; ++h2) {
                    const float4 x4 = qa[ib][h2], y4 = qp[ib][h2];
                    xv[4 * h2] = x4.x; xv[4 * h2 + 1] = x4.y; xv[4 * h2 + 2] = x4.z; xv[4 * h2 + 3] = x4.w;
                    xpv[4 * h2] = y4.x; xpv[4 * h2 + 1] = y4.y; xpv[4 * h2 + 2] = y4.z; xpv[4 * h2 + 3] = y4.w;
                }
#pragma unroll
                for (int h4 = 0; h4 < 4; ++h4) {
                    const float4 c4 = rc[ib][h4];
                    cv[2 * h4] = c4.x; sv[2 * h4] = c4.y; cv[2 * h4 + 1] = c4.z; sv[2 * h4 + 1] = c4.w;
                }
                uint16_t hb[8], rb[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    float y = 0.f;
                    if (ok) y = lo_half ? (xv[e] * cv[e] - xpv[e] * sv[e]) : (xv[e] * cv[e] + xpv[e] * sv[e]);
                    if constexpr (REC) if (ok) a.dbg_q[((size_t)m * Hq + h) * D + d0 + e] = y;
                    y *= a.qscale;
                    hb[e] = kv_round<KVDT>(y);
                    rb[e] = kv_round<KVDT>(y - kv_float<KVDT>(hb[e]));
                }
#pragma unroll
                for (int w2 = 0; w2 < 4; ++w2) {
                    qh[u][ib][w2] = (uint32_t)hb[2 * w2] | ((uint32_t)hb[2 * w2 + 1] << 16);
                    qr[u][ib][w2] = (uint32_t)rb[2 * w2] | ((uint32_t)rb[2 * w2 + 1] << 16);
                }
            }
            mrun[u] = -INFINITY;
            lsum[u] = 0.f;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) o[u][mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }

        for (c0 = j0; c0 < j1; c0 += ACH) {
        c1 = min(j1, c0 + ACH);
        if (qg != 0 || c0 != j0) {                           // (the first chunk was staged above)
            __syncthreads();                                 // the previous chunk's entries are no longer read
            for (int x = tid; x < c1 - c0; x += 256) {
                const int j = c0 + x;
                smk[x] = mask[j];
                stab[x] = j < P ? tab[j] : (int16_t)b;
            }
            __syncthreads();
            fetch(0, qg == 0 && !a.no_append);
        }
        const int nsteps = (c1 - c0 + AK - 1) / AK;
        stash(0);
        __syncthreads();
        for (int st = 0; st < nsteps; ++st) {
            const int buf = st & 1;
            if (st + 1 < nsteps) fetch((st + 1) * AK, qg == 0 && !a.no_append);   // next step's loads fly during this one
            // the lane's 8 keys: step key 4 lg + e (e < 4) or 16 + 4 lg + e - 4; visible ones as bits
            const int kbase = c0 + st * AK + 4 * lg;
            uint32_t vbits = 0u;
            {
                // mask bytes of keys 4 lg + 0..3 and 16 + 4 lg + 0..3 as two aligned words
                const uint32_t w0 = *(const uint32_t*)&smk[st * AK + 4 * lg];
                const uint32_t w1 = *(const uint32_t*)&smk[st * AK + 16 + 4 * lg];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int ko = (e < 4) ? e : 12 + e;
                    const uint32_t byte = ((e < 4 ? w0 : w1) >> (8 * (e & 3))) & 0xFFu;
                    vbits |= ((kbase + ko < c1 && byte != 0u) ? 1u : 0u) << e;
                }
            }
#pragma unroll
            for (int u = 0; u < QTW; ++u) {
                if (qg + wave + 4 * u >= nqt) continue;      // wave-uniform
                f32x4_t s0 = f32x4_t{0.f, 0.f, 0.f, 0.f}, s1 = s0;
                u32x4 kf0[DB], kf1[DB];                      // every key fragment of the step in flight at once
#pragma unroll
                for (int ib = 0; ib < DB; ++ib) {
                    const int c = 4 * ib + lg;
                    kf0[ib] = *(const u32x4*)&ks[buf][ql][8 * (c ^ (ql % NCH))];
                    kf1[ib] = *(const u32x4*)&ks[buf][16 + ql][8 * (c ^ ((16 + ql) % NCH))];
                }
#pragma unroll
                for (int ib = 0; ib < DB; ++ib) {
                    s0 = mma_kv<KVDT>(kf0[ib], qh[u][ib], s0);
                    s1 = mma_kv<KVDT>(kf1[ib], qh[u][ib], s1);
                    s0 = mma_kv<KVDT>(kf0[ib], qr[u][ib], s0);
                    s1 = mma_kv<KVDT>(kf1[ib], qr[u][ib], s1);
                }
                u32x4 vf[MB];                                // value fragments: read during the softmax
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) vf[mb] = *(const u32x4*)&vt[buf][16 * mb + ql][8 * lg];
                const int last = P + qtok[u] - kbase;         // keys up to kbase + last are causal
                float sv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int ko = (e < 4) ? e : 12 + e;
                    const float x = e < 4 ? s0[e] : s1[e - 4];
                    sv[e] = (((vbits >> e) & 1u) && ko <= last) ? x : -INFINITY;
                }
                if (rmask) {                                 // this query row's own mask (uniform branch)
                    const uint8_t* rrow = rmask + (size_t)min(qtok[u], n - 1) * rq.mask_len;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int j = min(kbase + ((e < 4) ? e : 12 + e), rq.mask_len - 1);
                        if (rrow[j] == 0) sv[e] = -INFINITY;
                    }
                }
                if constexpr (REC) {                             // test support: this tile's visible scores
                    const int r = 16 * (qg + wave + 4 * u) + ql;
                    if (r < R) {
                        const size_t row = ((size_t)(rowbase + r / gs) * Hq + g * gs + r % gs) * a.dbg_keys;
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const int j = kbase + ((e < 4) ? e : 12 + e);
                            if (sv[e] != -INFINITY && j < a.dbg_keys) a.dbg_logits[row + j] = sv[e] * 0.69314718055994531f;
                        }
                    }
                }
                float mx = sv[0];
#pragma unroll
                for (int e = 1; e < 8; ++e) mx = fmaxf(mx, sv[e]);
                float x0, x1;
                lane_pair_k(mx, 16, x0, x1);
                mx = fmaxf(x0, x1);
                lane_pair_k(mx, 32, x0, x1);
                mx = fmaxf(x0, x1);
                const float mn = fmaxf(mrun[u], mx);
                // no key seen yet (mn = -inf): base 0 makes every term and the correction 0
                const float base = mn == -INFINITY ? 0.f : mn;
                const float corr = __builtin_amdgcn_exp2f(mrun[u] - base);
                float pv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) pv[e] = __builtin_amdgcn_exp2f(sv[e] - base);
                float ps = 0.f;
#pragma unroll
                for (int e = 0; e < 8; ++e) ps += pv[e];
                lsum[u] = lsum[u] * corr + ps;
                mrun[u] = mn;
                u32x4 pb;
#pragma unroll
                for (int w2 = 0; w2 < 4; ++w2) pb[w2] = kv_pack2<KVDT>(pv[2 * w2], pv[2 * w2 + 1]);
                if (__any(corr != 1.f)) {                        // the running maximum moved in some lane
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                        for (int jj = 0; jj < 4; ++jj) o[u][mb][jj] *= corr;
                }
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) o[u][mb] = mma_kv<KVDT>(vf[mb], pb, o[u][mb]);
            }
            if (st + 1 < nsteps) stash(buf ^ 1);
            __syncthreads();
        }
        }

        // ---- this split's partial of each query vector: (max, sum, unnormalized output)
#pragma unroll
        for (int u = 0; u < QTW; ++u) {
            const int qt = qg + wave + 4 * u;
            if (qt >= nqt) continue;
            float x0, x1, lt = lsum[u];
            lane_pair_k(lt, 16, x0, x1);
            lt = x0 + x1;
            lane_pair_k(lt, 32, x0, x1);
            lt = x0 + x1;
            const int r = 16 * qt + ql;
            if (r >= R) continue;
            const int i = r / gs, h = g * gs + (r % gs);
            const int m = rowbase + i;
            float* pp = a.part + (((size_t)m * Hq + h) * a.nsplit_max + split) * (D + 2);
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) pp[2 + 16 * mb + 4 * lg + jj] = o[u][mb][jj];
            if (lg == 0) {
                pp[0] = mrun[u];
                pp[1] = lt;
            }
        }
    }
}

// ------------------------------------------------------------------ matrix-core attention, cache rows by direct loads
//
// attn_mma_kernel for items of at most 256 query vectors per kv head (up to four
// tiles per wave), with the same split, step order, arithmetic and partials
// (results are bitwise equal), but with the cache rows of each 32-key step
// brought into LDS by direct-to-LDS buffer loads issued ATTN_NB - 1 steps ahead
// instead of through registers one step ahead.  A key the split does not keep (masked,
// past the split, or a row of this forward, which is written in afterwards)
// is read at an offset past the buffer's end, which the hardware answers with
// zeros without a memory access.  K and V are stored as in memory, 16-byte
// chunk c of key k at position c ^ (k mod chunks per row); the value fragments
// of O^T += V^T P^T come from ds_read_b64_tr_b16, which hands lane i of each
// 16-lane group element i mod 4 of the 8 bytes read by lane 4 e + i / 4 of the
// group, as element e (e < 4): the four keys of a fragment half become one
// lane's four k slots.  The whole split's table entries and mask bytes (at
// most ATTN_SCH keys) and the rows of a per-query-row mask (at most ATTN_RSM
// bytes) are staged first; LDS is read through inline assembly and the
// workgroup synchronizes with a bare s_barrier, so no compiler-inserted wait
// drains the loads in flight.
constexpr int ATTN_NB = 4;                // step buffers (K and V of 32 keys each)
constexpr int ATTN_SCH = 1024;            // most keys of one split on this path
constexpr int ATTN_RSM = 8192;            // bytes of per-query-row mask staged per split (rows x split keys)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t attn_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ void attn_dma(__amdgpu_buffer_rsrc_t r, uint32_t off, void* lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, off, 0, 0, 2 /* nt */);
}
__device__ __forceinline__ u32x4 attn_lds16(uint32_t a) {
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a));
    return v;
}
__device__ __forceinline__ u32x2 attn_lds_tr(uint32_t a) {
    u32x2 v;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(a));
    return v;
}
__device__ __forceinline__ uint32_t attn_lds4(uint32_t a) {
    uint32_t v;
    asm volatile("ds_read_b32 %0, %1" : "=v"(v) : "v"(a));
    return v;
}
__device__ __forceinline__ uint32_t attn_lds_u16(uint32_t a) {
    uint32_t v;
    asm volatile("ds_read_u16 %0, %1" : "=v"(v) : "v"(a));
    return v;
}
__device__ __forceinline__ uint32_t attn_lds_u8(uint32_t a) {
    uint32_t v;
    asm volatile("ds_read_u8 %0, %1" : "=v"(v) : "v"(a));
    return v;
}
__device__ __forceinline__ void attn_lgkm() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// After attn_lgkm: makes v depend on the wait, so no use of a value read by
// inline assembly moves above it (the compiler takes such values as ready).
__device__ __forceinline__ void touch_v(u32x4& v) { asm volatile("" : "+v"(v)); }
__device__ __forceinline__ void touch_u(uint32_t& v) { asm volatile("" : "+v"(v)); }
template <int N>
__device__ __forceinline__ void attn_vm() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }
__device__ __forceinline__ void attn_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// QTW: query tiles of 16 vectors per wave (1, 2 or 4; tile wave + 4 u); with
// more than one, one workgroup per CU holds their registers.
template <int D, int KVDT, int QTW, bool REC = false>
__global__ __launch_bounds__(256, QTW == 1 ? 2 : 1) void attn_dma_kernel(AttnArgs a) {
    constexpr int HALF = D / 2;
    constexpr int NCH = D / 8;               // 16-byte chunks per cache row
    constexpr int DB = D / 32;               // k-blocks of the score products
    constexpr int MB = D / 16;               // row blocks of O^T
    constexpr int RB = 2 * D;                // bytes per cache row
    constexpr int SB = AK * RB;              // bytes of one step's K (or V)
    constexpr int KPI = 1024 / RB;           // keys per direct load (64 lanes x 16 bytes)
    constexpr int NI = SB / 1024 / 4;        // direct loads per wave per step, K and V each
    constexpr int VMN = 2 * NI * (ATTN_NB - 2);   // loads a lane may leave in flight at the top of a step
    static_assert(NI >= 1 && VMN <= 63, "step geometry");
    static_assert(AK * NCH % 256 == 0, "new-row staging");
    __shared__ __attribute__((aligned(16))) uint8_t kvs[ATTN_NB][2][SB];
    __shared__ int16_t stab[ATTN_SCH];
    __shared__ __attribute__((aligned(16))) uint8_t smk[ATTN_SCH];
    __shared__ __attribute__((aligned(16))) uint8_t srm[ATTN_RSM];   // [row][split key] when the request has row masks

    const int item = blockIdx.x, g = blockIdx.y, split = blockIdx.z;
    const ItemDev it = a.meta.items[item];
    const ReqDev rq = it.rq;
    const int b = it.slot;
    const int P = rq.P, n = rq.n;
    const int L = P + n;
    int split_len = max(ATTN_MIN_SPLIT, (L + rq.splits - 1) / rq.splits);
    split_len = (split_len + KGROUPS - 1) / KGROUPS * KGROUPS;
    const int nsplit = (L + split_len - 1) / split_len;
    if (split >= nsplit) return;
    const int j0 = split * split_len, j1 = min(L, j0 + split_len);

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ql = lane & 15, lg = lane >> 4;
    const int Hq = a.Hq, Hkv = a.Hkv;
    const int gs = Hq / Hkv;
    const int R = gs * n;
    const int nqt = (R + 15) / 16;
    const size_t lstride = (size_t)rq.S * Hkv * rq.cap * D;
    uint16_t* kl = rq.kc + (size_t)a.layer * lstride;
    uint16_t* vl = rq.vc + (size_t)a.layer * lstride;
    const uint8_t* mask = a.meta.masks + rq.mask_off + (size_t)b * rq.mask_len;
    const int16_t* tab = rq.table + (size_t)b * rq.cap;
    const int rowbase = rq.row0 + b * n;

    // ---- the split's table entries and mask bytes (and each query row's own mask)
    for (int x = tid; x < j1 - j0; x += 256) {
        const int j = j0 + x;
        smk[x] = mask[j];
        stab[x] = j < P ? tab[j] : (int16_t)b;
    }
    const uint8_t* rmask = rq.rowmask_off >= 0 ? a.meta.masks + rq.rowmask_off + (size_t)b * n * rq.mask_len : nullptr;
    const int rspan = (j1 - j0 + 3) & ~3;                    // row stride of srm (the host checked n * rspan fits)
    if (rmask)
        for (int q = tid; q < n * rspan; q += 256) {
            const int i = q / rspan, x = q - i * rspan;
            srm[q] = x < j1 - j0 ? rmask[(size_t)i * rq.mask_len + j0 + x] : (uint8_t)0;
        }
    __syncthreads();

    // ---- direct loads of step s into buffer s mod ATTN_NB: lane l of load h of
    // this wave carries chunk position l mod NCH of key (NI wave + h) KPI + l / NCH
    const int nsteps = (j1 - j0 + AK - 1) / AK;
    const uint32_t lbytes = (uint32_t)(lstride * 2);
    const __amdgpu_buffer_rsrc_t rk = attn_rsrc(kl, lbytes), rv = attn_rsrc(vl, lbytes);
    const uint32_t smk_a = (uint32_t)(uintptr_t)smk, stab_a = (uint32_t)(uintptr_t)stab;
    const uint32_t kvs_a = (uint32_t)(uintptr_t)&kvs[0][0][0];
    const int cstop = min(j1, P);                            // keys below this come from the cache
    auto issue = [&](int s) {
        uint32_t off[NI];
#pragma unroll
        for (int h = 0; h < NI; ++h) {
            const int key = (NI * wave + h) * KPI + lane / NCH;
            const int x = min(s * AK + key, ATTN_SCH - 1), j = j0 + s * AK + key;
            uint32_t mk = attn_lds_u8(smk_a + (uint32_t)x);
            uint32_t tb = attn_lds_u16(stab_a + 2u * (uint32_t)x);
            attn_lgkm();
            touch_u(mk);
            touch_u(tb);
            const int slot = (int)(int16_t)tb;
            const int c = (lane % NCH) ^ (key % NCH);
            const bool kept = s < nsteps && j < cstop && mk != 0u;
            off[h] = kept ? (uint32_t)(((((size_t)slot * Hkv + g) * rq.cap + j) * D + 8 * c) * 2) : 0xFFFFFFF0u;
        }
        uint8_t* kb = &kvs[s % ATTN_NB][0][0];
#pragma unroll
        for (int h = 0; h < NI; ++h) {
            const int blk = (NI * wave + h) * 1024;
            attn_dma(rk, off[h], kb + blk);
            attn_dma(rv, off[h], kb + SB + blk);
        }
    };
#pragma unroll
    for (int s = 0; s < ATTN_NB - 1; ++s) issue(s);

    // ---- this wave's query tiles: rotated, scaled, split into rounded part and residual
    const bool active = wave < nqt;
    u32x4 qh[QTW][DB], qr[QTW][DB];
    int qtok[QTW];
    float mrun[QTW], lsum[QTW];
    f32x4_t o[QTW][MB];
#pragma unroll
    for (int u = 0; u < QTW; ++u) {
        const int r = 16 * (wave + 4 * u) + ql;
        const bool ok = wave + 4 * u < nqt && r < R;
        const int i = ok ? r / gs : 0, h = g * gs + (ok ? r % gs : 0);
        const int m = rowbase + i;
        const float* qrow = a.qkv + (size_t)m * a.qkv_ld + (size_t)h * D;
        qtok[u] = ok ? i : n;
        mrun[u] = -INFINITY;
        lsum[u] = 0.f;
        // every load of the tile at once (row 0 of the item stands in for a missing
        // row): q and its rotary partners, then (cos, sin) at the row's position
        float4 qa[DB][2], qp[DB][2], rc[DB][4];
#pragma unroll
        for (int ib = 0; ib < DB; ++ib) {
            const int d0 = 32 * ib + 8 * lg;
            const bool lo_half = d0 < HALF;
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                qa[ib][h2] = ((const float4*)(qrow + d0))[h2];
                qp[ib][h2] = ((const float4*)(qrow + (lo_half ? d0 + HALF : d0 - HALF)))[h2];
            }
        }
        const int pos = a.meta.positions[m];
#pragma unroll
        for (int ib = 0; ib < DB; ++ib) {
            const int d0 = 32 * ib + 8 * lg;
            const float4* r4 = (const float4*)(a.rope + (size_t)pos * HALF + (d0 < HALF ? d0 : d0 - HALF));
#pragma unroll
            for (int h4 = 0; h4 < 4; ++h4) rc[ib][h4] = r4[h4];
        }
#pragma unroll
        for (int ib = 0; ib < DB; ++ib) {
            // dims d0 .. d0 + 7 lie in one rotary half
            const int d0 = 32 * ib + 8 * lg;
            const bool lo_half = d0 < HALF;
            float xv[8], xpv[8], cv[8], sv[8];
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const float4 x4 = qa[ib][h2], y4 = qp[ib][h2];
                xv[4 * h2] = x4.x; xv[4 * h2 + 1] = x4.y; xv[4 * h2 + 2] = x4.z; xv[4 * h2 + 3] = x4.w;
                xpv[4 * h2] = y4.x; xpv[4 * h2 + 1] = y4.y; xpv[4 * h2 + 2] = y4.z; xpv[4 * h2 + 3] = y4.w;
            }
#pragma unroll
            for (int h4 = 0; h4 < 4; ++h4) {
                const float4 c4 = rc[ib][h4];
                cv[2 * h4] = c4.x; sv[2 * h4] = c4.y; cv[2 * h4 + 1] = c4.z; sv[2 * h4 + 1] = c4.w;
            }
            uint16_t hb[8], rb[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float y = 0.f;
                if (ok) y = lo_half ? (xv[e] * cv[e] - xpv[e] * sv[e]) : (xv[e] * cv[e] + xpv[e] * sv[e]);
                if constexpr (REC) if (ok) a.dbg_q[((size_t)m * Hq + h) * D + d0 + e] = y;
                y *= a.qscale;
                hb[e] = kv_round<KVDT>(y);
                rb[e] = kv_round<KVDT>(y - kv_float<KVDT>(hb[e]));
            }
#pragma unroll
            for (int w2 = 0; w2 < 4; ++w2) {
                qh[u][ib][w2] = (uint32_t)hb[2 * w2] | ((uint32_t)hb[2 * w2 + 1] << 16);
                qr[u][ib][w2] = (uint32_t)rb[2 * w2] | ((uint32_t)rb[2 * w2 + 1] << 16);
            }
        }
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) o[u][mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    for (int st = 0; st < nsteps; ++st) {
        const int buf = st % ATTN_NB;
        if constexpr (REC) attn_vm<0>();                     // the record's stores share the load counter
        else attn_vm<VMN>();                                 // this step's loads (later steps may stay in flight)
        attn_barrier();                                      // every lane's loads of this step are in LDS
        issue(st + ATTN_NB - 1);                             // into the buffer every wave finished with
        const int x0 = st * AK;
        if (j0 + x0 + AK > P && j0 + x0 < j1) {              // the step holds rows of this forward (uniform)
            uint8_t* kb = &kvs[buf][0][0];
#pragma unroll
            for (int u = 0; u < AK * NCH / 256; ++u) {
                const int q = tid + 256 * u, k = q / NCH, c = q % NCH;
                const int j = j0 + x0 + k;
                if (j < P || j >= j1) continue;
                const int i = j - P;
                const int m = rowbase + i;
                const int pos = a.meta.positions[m];
                const float* krow = a.qkv + (size_t)m * a.qkv_ld + (size_t)(Hq + g) * D;
                const float* vrow = a.qkv + (size_t)m * a.qkv_ld + (size_t)(Hq + Hkv + g) * D;
                uint16_t kb8[8], vb8[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int d = 8 * c + e;
                    const bool lo_half = d < HALF;
                    const float xk = krow[d];
                    const float xp = lo_half ? krow[d + HALF] : krow[d - HALF];
                    const float2 cs = a.rope[(size_t)pos * HALF + (lo_half ? d : d - HALF)];
                    const float y = lo_half ? (xk * cs.x - xp * cs.y) : (xk * cs.x + xp * cs.y);
                    kb8[e] = kv_round<KVDT>(y);
                    vb8[e] = kv_round<KVDT>(vrow[d]);
                }
                u32x4 kk, vv;
#pragma unroll
                for (int w2 = 0; w2 < 4; ++w2) {
                    kk[w2] = (uint32_t)kb8[2 * w2] | ((uint32_t)kb8[2 * w2 + 1] << 16);
                    vv[w2] = (uint32_t)vb8[2 * w2] | ((uint32_t)vb8[2 * w2 + 1] << 16);
                }
                if (!a.no_append) {                          // append: owner of row j writes it
                    const size_t off = (((size_t)b * Hkv + g) * rq.cap + j) * D + 8 * c;
                    *(u32x4*)(kl + off) = kk;
                    *(u32x4*)(vl + off) = vv;
                    if (a.layer == 0 && g == 0 && c == 0) rq.table[(size_t)b * rq.cap + j] = (int16_t)b;
                }
                if (smk[x0 + k] != 0) {                      // a kept row enters; a dropped one stays zero
                    const int pos16 = 16 * (c ^ (k % NCH));
                    *(u32x4*)(kb + k * RB + pos16) = kk;
                    *(u32x4*)(kb + SB + k * RB + pos16) = vv;
                }
            }
            attn_barrier();
        }
        if (active) {
            const uint32_t kb_a = kvs_a + (uint32_t)(buf * 2 * SB), vb_a = kb_a + SB;
            const int kbase = j0 + x0 + 4 * lg;
            u32x4 kf0[DB], kf1[DB], vf[MB];
#pragma unroll
            for (int ib = 0; ib < DB; ++ib) {
                const int c = 4 * ib + lg;
                kf0[ib] = attn_lds16(kb_a + (uint32_t)(ql * RB + 16 * (c ^ (ql % NCH))));
                kf1[ib] = attn_lds16(kb_a + (uint32_t)((16 + ql) * RB + 16 * (c ^ ((16 + ql) % NCH))));
            }
            // value fragments: read h gives keys 16 h + 4 lg + e; this lane supplies
            // key 16 h + 4 lg + ql / 4, dims 16 mb + 4 (ql mod 4) .. + 3
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                u32x2 p0, p1;
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    const int key = 16 * hh + 4 * lg + (ql >> 2);
                    const int d = 16 * mb + 4 * (ql & 3);
                    const uint32_t ad = vb_a + (uint32_t)(key * RB + 16 * ((d >> 3) ^ (key % NCH)) + 2 * (d & 7));
                    if (hh == 0) p0 = attn_lds_tr(ad);
                    else p1 = attn_lds_tr(ad);
                }
                vf[mb] = u32x4{p0[0], p0[1], p1[0], p1[1]};
            }
            uint32_t w0 = attn_lds4(smk_a + (uint32_t)(x0 + 4 * lg));
            uint32_t w1 = attn_lds4(smk_a + (uint32_t)(x0 + 16 + 4 * lg));
            attn_lgkm();
            touch_u(w0);
            touch_u(w1);
#pragma unroll
            for (int ib = 0; ib < DB; ++ib) { touch_v(kf0[ib]); touch_v(kf1[ib]); }
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) touch_v(vf[mb]);
            uint32_t vb0 = 0u;                               // keys of the step this split keeps
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int ko = (e < 4) ? e : 12 + e;
                const uint32_t byte = ((e < 4 ? w0 : w1) >> (8 * (e & 3))) & 0xFFu;
                vb0 |= ((kbase + ko < j1 && byte != 0u) ? 1u : 0u) << e;
            }
#pragma unroll
            for (int u = 0; u < QTW; ++u) {
                if (wave + 4 * u >= nqt) continue;           // wave-uniform
                uint32_t vbits = vb0;
                if (rmask) {                                 // this query row's own mask bytes (uniform branch)
                    const uint32_t ra = (uint32_t)(uintptr_t)srm + (uint32_t)(min(qtok[u], n - 1) * rspan + x0 + 4 * lg);
                    uint32_t r0 = attn_lds4(ra), r1 = attn_lds4(ra + 16);
                    attn_lgkm();
                    touch_u(r0);
                    touch_u(r1);
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if ((((e < 4 ? r0 : r1) >> (8 * (e & 3))) & 0xFFu) == 0u) vbits &= ~(1u << e);
                }
                f32x4_t s0 = f32x4_t{0.f, 0.f, 0.f, 0.f}, s1 = s0;
#pragma unroll
                for (int ib = 0; ib < DB; ++ib) {
                    s0 = mma_kv<KVDT>(kf0[ib], qh[u][ib], s0);
                    s1 = mma_kv<KVDT>(kf1[ib], qh[u][ib], s1);
                    s0 = mma_kv<KVDT>(kf0[ib], qr[u][ib], s0);
                    s1 = mma_kv<KVDT>(kf1[ib], qr[u][ib], s1);
                }
                const int last = P + qtok[u] - kbase;        // keys up to kbase + last are causal
                float sv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int ko = (e < 4) ? e : 12 + e;
                    const float x = e < 4 ? s0[e] : s1[e - 4];
                    sv[e] = (((vbits >> e) & 1u) && ko <= last) ? x : -INFINITY;
                }
                if constexpr (REC) {                         // test support: this tile's visible scores
                    const int r = 16 * (wave + 4 * u) + ql;
                    if (r < R) {
                        const size_t row = ((size_t)(rowbase + r / gs) * Hq + g * gs + r % gs) * a.dbg_keys;
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const int j = kbase + ((e < 4) ? e : 12 + e);
                            if (sv[e] != -INFINITY && j < a.dbg_keys) a.dbg_logits[row + j] = sv[e] * 0.69314718055994531f;
                        }
                    }
                }
                float mx = sv[0];
#pragma unroll
                for (int e = 1; e < 8; ++e) mx = fmaxf(mx, sv[e]);
                float x0f, x1f;
                lane_pair_k(mx, 16, x0f, x1f);
                mx = fmaxf(x0f, x1f);
                lane_pair_k(mx, 32, x0f, x1f);
                mx = fmaxf(x0f, x1f);
                const float mn = fmaxf(mrun[u], mx);
                // no key seen yet (mn = -inf): base 0 makes every term and the correction 0
                const float base = mn == -INFINITY ? 0.f : mn;
                const float corr = __builtin_amdgcn_exp2f(mrun[u] - base);
                float pv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) pv[e] = __builtin_amdgcn_exp2f(sv[e] - base);
                float ps = 0.f;
#pragma unroll
                for (int e = 0; e < 8; ++e) ps += pv[e];
                lsum[u] = lsum[u] * corr + ps;
                mrun[u] = mn;
                u32x4 pb;
#pragma unroll
                for (int w2 = 0; w2 < 4; ++w2) pb[w2] = kv_pack2<KVDT>(pv[2 * w2], pv[2 * w2 + 1]);
                if (__any(corr != 1.f)) {                    // the running maximum moved in some lane
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                        for (int jj = 0; jj < 4; ++jj) o[u][mb][jj] *= corr;
                }
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) o[u][mb] = mma_kv<KVDT>(vf[mb], pb, o[u][mb]);
            }
        }
    }
    attn_vm<0>();                                            // no direct load may land after the workgroup ends

    // ---- this split's partial of each query vector: (max, sum, unnormalized output)
#pragma unroll
    for (int u = 0; u < QTW; ++u) {
        if (wave + 4 * u >= nqt) continue;
        float x0f, x1f, lt = lsum[u];
        lane_pair_k(lt, 16, x0f, x1f);
        lt = x0f + x1f;
        lane_pair_k(lt, 32, x0f, x1f);
        lt = x0f + x1f;
        const int r = 16 * (wave + 4 * u) + ql;
        if (r < R) {
            const int i = r / gs, h = g * gs + (r % gs);
            const int m = rowbase + i;
            float* pp = a.part + (((size_t)m * Hq + h) * a.nsplit_max + split) * (D + 2);
            // 16-byte stores (the record is only 8-byte aligned; the hardware takes
            // 4-byte aligned wide stores): a store per value lengthens the launch's drain
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) __builtin_memcpy(pp + 2 + 16 * mb + 4 * lg, &o[u][mb], 16);
            if (lg == 0) {
                const float2 ml = {mrun[u], lt};
                __builtin_memcpy(pp, &ml, 8);
            }
        }
    }
}

hipError_t launch_attention(const AttnArgs& a, int head_dim, int queries_per_item_max, hipStream_t st) {
    const dim3 grid(a.meta.n_items, a.Hkv, a.nsplit_max), block(256);
    const dim3 mgrid(a.meta.M, a.Hq);
    const bool wide = queries_per_item_max > 4;
    const bool bf = a.kv_dt == DT_BF16;
    const bool one = queries_per_item_max <= 64;                // every item's query tiles: one per wave
    // the direct-load form takes up to four tiles per wave (256 query vectors per kv head)
    const int dq = !a.dma || queries_per_item_max > 256 ? 0 : one ? 1 : queries_per_item_max <= 128 ? 2 : 4;
#define ATTN_DMA_Q(D_, T_, R_)                                                                    \
    do {                                                                                          \
        if (bf) attn_dma_kernel<D_, DT_BF16, T_, R_><<<grid, block, 0, st>>>(a);                  \
        else attn_dma_kernel<D_, DT_F16, T_, R_><<<grid, block, 0, st>>>(a);                      \
    } while (0)
#define ATTN_MMA_R(D_, R_)                                                                        \
    do {                                                                                          \
        if (dq == 1) ATTN_DMA_Q(D_, 1, R_);                                                       \
        else if (dq == 2) ATTN_DMA_Q(D_, 2, R_);                                                  \
        else if (dq == 4) ATTN_DMA_Q(D_, 4, R_);                                                  \
        else if (bf && one) attn_mma_kernel<D_, DT_BF16, 1, R_><<<grid, block, 0, st>>>(a);       \
        else if (bf) attn_mma_kernel<D_, DT_BF16, 2, R_><<<grid, block, 0, st>>>(a);              \
        else if (one) attn_mma_kernel<D_, DT_F16, 1, R_><<<grid, block, 0, st>>>(a);              \
        else attn_mma_kernel<D_, DT_F16, 2, R_><<<grid, block, 0, st>>>(a);                       \
    } while (0)
#define ATTN_MMA(D_)                                                                              \
    do {                                                                                          \
        if (a.dbg_logits) ATTN_MMA_R(D_, true);          /* test support: record queries and scores */ \
        else ATTN_MMA_R(D_, false);                                                               \
    } while (0)
    if (head_dim == 128) {
        if (!a.vector_path) ATTN_MMA(128);
        else if (wide) attn_kernel<128, 8><<<grid, block, 0, st>>>(a);
        else attn_kernel<128, 4><<<grid, block, 0, st>>>(a);
        attn_merge_kernel<128><<<mgrid, dim3(128), 0, st>>>(a);
    } else if (head_dim == 64) {
        if (!a.vector_path) ATTN_MMA(64);
        else if (wide) attn_kernel<64, 8><<<grid, block, 0, st>>>(a);
        else attn_kernel<64, 4><<<grid, block, 0, st>>>(a);
        attn_merge_kernel<64><<<mgrid, dim3(64), 0, st>>>(a);
    } else {
        return hipErrorInvalidValue;
    }
#undef ATTN_MMA
#undef ATTN_MMA_R
#undef ATTN_DMA_Q
    return hipGetLastError();
}

// ------------------------------------------------------------------ fill

// p[0 .. n) = v.
__global__ __launch_bounds__(256) void fill_u32_kernel(uint32_t* __restrict__ p, size_t n, uint32_t v) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t v, hipStream_t st) {
    if (n == 0) return hipSuccess;
    const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 4096);
    fill_u32_kernel<<<blocks, 256, 0, st>>>(p, n, v);
    return hipGetLastError();
}

// ------------------------------------------------------------------ KV state kernels

__global__ void table_gather_kernel(const int16_t* __restrict__ src, int16_t* __restrict__ dst, const int* __restrict__ beam,
                                    int S, int cap, int P) {
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= (size_t)S * P) return;
    const int b = (int)(idx / P), j = (int)(idx % P);
    dst[(size_t)b * cap + j] = src[(size_t)beam[b] * cap + j];
}

hipError_t launch_table_gather(const int16_t* src, int16_t* dst, const int* beam, int S, int cap, int P, hipStream_t st) {
    const size_t n = (size_t)S * P;
    if (n == 0) return hipSuccess;
    table_gather_kernel<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st>>>(src, dst, beam, S, cap, P);
    return hipGetLastError();
}

// Rows [L][S][Hkv][n][D] of k, v to physical rows P..P+n-1 of every slot; the
// slots' table entries there become their own index.  One thread moves 16
// bytes of K and of V (D is a multiple of 8).
__global__ __launch_bounds__(256) void kv_append_kernel(uint16_t* __restrict__ kc, uint16_t* __restrict__ vc,
                                                        int16_t* __restrict__ table, const uint16_t* __restrict__ k,
                                                        const uint16_t* __restrict__ v, int L, int S, int Hkv, int cap, int D,
                                                        int P, int n) {
    const int tpr = D / 8;
    const size_t total = (size_t)L * S * Hkv * n * tpr;
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= total) return;
    size_t rem = idx;
    const int e = (int)(rem % tpr); rem /= tpr;
    const int i = (int)(rem % n); rem /= n;
    const int g = (int)(rem % Hkv); rem /= Hkv;
    const int b = (int)(rem % S); rem /= S;
    const int l = (int)rem;
    const size_t dst = ((((size_t)l * S + b) * Hkv + g) * cap + (P + i)) * D + 8 * e;
    *(uint4*)(kc + dst) = *(const uint4*)(k + 8 * idx);
    *(uint4*)(vc + dst) = *(const uint4*)(v + 8 * idx);
    if (l == 0 && g == 0 && e == 0) table[(size_t)b * cap + P + i] = (int16_t)b;
}

hipError_t launch_kv_append(uint16_t* kc, uint16_t* vc, int16_t* table, const uint16_t* k, const uint16_t* v,
                            int L, int S, int Hkv, int cap, int D, int P, int n, hipStream_t st) {
    if (D % 8) return hipErrorInvalidValue;
    const size_t total = (size_t)L * S * Hkv * n * (D / 8);
    if (total == 0) return hipSuccess;
    kv_append_kernel<<<dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st>>>(kc, vc, table, k, v, L, S, Hkv, cap, D, P, n);
    return hipGetLastError();
}

__global__ void kv_read_kernel(const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc, const int16_t* __restrict__ table,
                               int layer, int slot, int start, int count, int S, int Hkv, int cap, int D,
                               uint16_t* __restrict__ k_out, uint16_t* __restrict__ v_out) {
    const size_t total = (size_t)Hkv * count * D;
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const int d = (int)(idx % D);
    const int c = (int)((idx / D) % count);
    const int g = (int)(idx / ((size_t)D * count));
    const int j = start + c;
    const int ps = table[(size_t)slot * cap + j];
    const size_t src = ((((size_t)layer * S + ps) * Hkv + g) * cap + j) * D + d;
    k_out[idx] = kc[src];
    v_out[idx] = vc[src];
}

hipError_t launch_kv_read(const uint16_t* kc, const uint16_t* vc, const int16_t* table, int layer, int slot,
                          int start, int count, int S, int Hkv, int cap, int D, uint16_t* k_out, uint16_t* v_out,
                          hipStream_t st) {
    const size_t total = (size_t)Hkv * count * D;
    if (total == 0) return hipSuccess;
    kv_read_kernel<<<dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st>>>(kc, vc, table, layer, slot, start, count,
                                                                                  S, Hkv, cap, D, k_out, v_out);
    return hipGetLastError();
}

// ------------------------------------------------------------------ compaction and capture

// dst row i of slot b (for every layer and kv head) = the row src[b][i] of the
// slot's view, read through the beam table (physical slot table[b][j] holds
// row j); src[b][i] < 0 writes a zero row.  One thread moves 16 bytes of K and
// 16 of V; a row is D / 8 consecutive threads, so a wave's loads and stores
// cover whole rows.  dst rows of one (layer, slot, kv head) are dst_stride
// rows apart.
__global__ __launch_bounds__(256) void kv_gather_rows_kernel(const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
                                                             const int16_t* __restrict__ table, const int* __restrict__ src,
                                                             int L, int S, int Hkv, int cap, int D, int Pn, int dst_stride,
                                                             uint16_t* __restrict__ k_dst, uint16_t* __restrict__ v_dst) {
    const int tpr = D / 8;
    const size_t rows = (size_t)L * S * Hkv * Pn;
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= rows * tpr) return;
    const int e = (int)(idx % tpr);
    size_t r = idx / tpr;
    const int i = (int)(r % Pn); r /= Pn;
    const int g = (int)(r % Hkv); r /= Hkv;
    const int b = (int)(r % S);
    const int l = (int)(r / S);
    const size_t dst = ((((size_t)l * S + b) * Hkv + g) * dst_stride + i) * D + 8 * e;
    const int j = src[(size_t)b * Pn + i];
    uint4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
    if (j >= 0) {
        const int ps = table[(size_t)b * cap + j];
        const size_t so = ((((size_t)l * S + ps) * Hkv + g) * cap + j) * D + 8 * e;
        kv = *(const uint4*)(kc + so);
        vv = *(const uint4*)(vc + so);
    }
    *(uint4*)(k_dst + dst) = kv;
    *(uint4*)(v_dst + dst) = vv;
}

hipError_t launch_kv_gather_rows(const uint16_t* kc, const uint16_t* vc, const int16_t* table, const int* src, int L, int S,
                                 int Hkv, int cap, int D, int Pn, int dst_stride, uint16_t* k_dst, uint16_t* v_dst,
                                 hipStream_t st) {
    if (D % 8) return hipErrorInvalidValue;
    const size_t n = (size_t)L * S * Hkv * Pn * (D / 8);
    if (n == 0) return hipSuccess;
    kv_gather_rows_kernel<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st>>>(kc, vc, table, src, L, S, Hkv, cap, D,
                                                                                    Pn, dst_stride, k_dst, v_dst);
    return hipGetLastError();
}

// In-place compaction of one cache (K or V): row i of slot b becomes the row
// src[b][i] of the slot's view (through the beam table), or zero where
// src[b][i] < 0.  src[b][i] >= i (kept rows in ascending order), so a row read
// for destination i is never a destination below i.  One workgroup owns one
// column slice (KC_SLICES per row) of one (layer, kv head, K or V) for every
// slot and walks the destination rows in chunks of `chunk` positions:
//  - all of a chunk's loads complete before any of its stores (the wait and
//    the barrier before the stores);
//  - the loads of chunk c + 1 are issued before the stores of chunk c: they
//    read rows at or above the first position of chunk c + 1, the stores of
//    chunk c write rows below it, so the two never touch the same element;
//  - rows read by later chunks lie at or above their destinations, above
//    every row written so far.
// So no element is overwritten before every read of it.  Column slices are
// independent (a row's slice moves with the row).
constexpr int KC_THREADS = 512;
constexpr int KC_PIECES = 4;
constexpr int KC_SLICES = 2;

struct KcChunk {
    uint4 v[KC_PIECES];
};

__device__ __forceinline__ void kc_load(const uint16_t* c, const int16_t* __restrict__ table, const int* __restrict__ src,
                                        int l, int g, int S, int Hkv, int cap, int D, int Pn, int pps, int col0, int i0,
                                        int cn, KcChunk& ch) {
    const int pieces = S * cn * pps;
#pragma unroll
    for (int k = 0; k < KC_PIECES; ++k) {
        const int p = threadIdx.x + k * KC_THREADS;
        ch.v[k] = make_uint4(0u, 0u, 0u, 0u);
        if (p < pieces) {
            const int r = p / pps;
            const int b = r / cn;
            const int i = i0 + r % cn;
            const int j = src[(size_t)b * Pn + i];
            if (j >= 0) {
                const int ps = table[(size_t)b * cap + j];
                ch.v[k] = *(const uint4*)(c + ((((size_t)l * S + ps) * Hkv + g) * cap + j) * D + col0 + 8 * (p % pps));
            }
        }
    }
}

__device__ __forceinline__ void kc_store(uint16_t* c, int l, int g, int S, int Hkv, int cap, int D, int pps, int col0,
                                         int i0, int cn, const KcChunk& ch) {
    const int pieces = S * cn * pps;
#pragma unroll
    for (int k = 0; k < KC_PIECES; ++k) {
        const int p = threadIdx.x + k * KC_THREADS;
        if (p < pieces) {
            const int r = p / pps;
            const int b = r / cn;
            const int i = i0 + r % cn;
            *(uint4*)(c + ((((size_t)l * S + b) * Hkv + g) * cap + i) * D + col0 + 8 * (p % pps)) = ch.v[k];
        }
    }
}

__global__ __launch_bounds__(KC_THREADS) void kv_compact_kernel(uint16_t* kc, uint16_t* vc, const int16_t* __restrict__ table,
                                                                const int* __restrict__ src, int S, int Hkv, int cap,
                                                                int D, int Pn, int chunk) {
    const int slice = blockIdx.x % KC_SLICES;
    const int u = blockIdx.x / KC_SLICES;
    const int l = u / (2 * Hkv);
    const int g = (u / 2) % Hkv;
    uint16_t* c = (u & 1) ? vc : kc;
    const int pps = D / 8 / KC_SLICES;                       // 16-byte pieces of a row slice
    const int col0 = slice * pps * 8;                        // first element of the slice
    KcChunk a, b;
    kc_load(c, table, src, l, g, S, Hkv, cap, D, Pn, pps, col0, 0, min(chunk, Pn), a);
    for (int i0 = 0; i0 < Pn; i0 += 2 * chunk) {
        // chunk at i0 (in a), then chunk at i0 + chunk (in b)
        const int i1 = i0 + chunk, i2 = i0 + 2 * chunk;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");     // this wave's accesses have completed
        __syncthreads();                                     // and so have every other wave's
        if (i1 < Pn) kc_load(c, table, src, l, g, S, Hkv, cap, D, Pn, pps, col0, i1, min(chunk, Pn - i1), b);
        kc_store(c, l, g, S, Hkv, cap, D, pps, col0, i0, min(chunk, Pn - i0), a);
        if (i1 >= Pn) break;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (i2 < Pn) kc_load(c, table, src, l, g, S, Hkv, cap, D, Pn, pps, col0, i2, min(chunk, Pn - i2), a);
        kc_store(c, l, g, S, Hkv, cap, D, pps, col0, i1, min(chunk, Pn - i1), b);
    }
}

hipError_t launch_kv_compact(uint16_t* kc, uint16_t* vc, const int16_t* table, const int* src, int L, int S, int Hkv,
                             int cap, int D, int Pn, hipStream_t st) {
    if (D % (8 * KC_SLICES)) return hipErrorInvalidValue;
    if (Pn == 0 || L == 0) return hipSuccess;
    const int pps = D / 8 / KC_SLICES;
    if ((long)S * pps > (long)KC_THREADS * KC_PIECES) return hipErrorInvalidValue;   // a chunk holds every slot's row
    const int chunk = KC_THREADS * KC_PIECES / (S * pps);
    kv_compact_kernel<<<dim3((unsigned)(L * Hkv * 2 * KC_SLICES)), dim3(KC_THREADS), 0, st>>>(kc, vc, table, src, S, Hkv,
                                                                                             cap, D, Pn, chunk);
    return hipGetLastError();
}

// ------------------------------------------------------------------ top-1 of the LM head

// One workgroup per row: the tiles' (max, index, sum of exp(v - max)) reduced
// in a fixed order (strided per thread, then a tree), so the result does not
// depend on timing.  Ties on the value take the smallest index.
__global__ __launch_bounds__(256) void top1_merge_kernel(const float4* __restrict__ part, int ntiles, int32_t* __restrict__ token,
                                                         float* __restrict__ p, float* __restrict__ logit) {
    __shared__ float smx[256];
    __shared__ int sarg[256];
    __shared__ float sse[256];
    const int m = blockIdx.x, tid = threadIdx.x;
    const float4* row = part + (size_t)m * ntiles;
    float mx = -INFINITY;
    int arg = INT_MAX;
    for (int t = tid; t < ntiles; t += 256) {
        const float4 e = row[t];
        const int ei = __float_as_int(e.y);
        if (e.x > mx || (e.x == mx && ei < arg)) {
            mx = e.x;
            arg = ei;
        }
    }
    smx[tid] = mx;
    sarg[tid] = arg;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) {
            const float x2 = smx[tid + o];
            const int a2 = sarg[tid + o];
            if (x2 > smx[tid] || (x2 == smx[tid] && a2 < sarg[tid])) {
                smx[tid] = x2;
                sarg[tid] = a2;
            }
        }
        __syncthreads();
    }
    const float gmx = smx[0];
    float se = 0.f;
    for (int t = tid; t < ntiles; t += 256) {
        const float4 e = row[t];
        se += e.z * expf(e.x - gmx);
    }
    sse[tid] = se;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) sse[tid] += sse[tid + o];
        __syncthreads();
    }
    if (tid == 0) {
        token[m] = sarg[0];
        p[m] = 1.0f / sse[0];
        if (logit) logit[m] = gmx;
    }
}

hipError_t launch_top1_merge(const float4* part, int M, int ntiles, int32_t* token, float* p, float* logit, hipStream_t st) {
    if (M < 1 || ntiles < 1) return hipErrorInvalidValue;
    top1_merge_kernel<<<dim3((unsigned)M), dim3(256), 0, st>>>(part, ntiles, token, p, logit);
    return hipGetLastError();
}

// ------------------------------------------------------------------ stage-0 embedding gather

// Row m of out = row ids[m] of the token table [vocab][row_elems], copied
// unchanged; an id outside [0, vocab) gives a zero row and sets *err.  One
// workgroup per row; T is the copy width (16 bytes when both pointers allow).
template <class T>
__global__ __launch_bounds__(256) void embed_gather_kernel(const T* __restrict__ table, const int32_t* __restrict__ ids,
                                                           int vocab, int row_elems, T* __restrict__ out,
                                                           unsigned* __restrict__ err) {
    const int m = blockIdx.x;
    const int id = ids[m];
    T* dst = out + (size_t)m * row_elems;
    if (id < 0 || id >= vocab) {
        for (int i = threadIdx.x; i < row_elems; i += 256) dst[i] = T(0);
        if (threadIdx.x == 0) atomicOr(err, 1u);
        return;
    }
    const T* src = table + (size_t)id * row_elems;
    for (int i = threadIdx.x; i < row_elems; i += 256) dst[i] = src[i];
}

hipError_t launch_embed_gather(const uint16_t* table, const int32_t* ids, int n, int vocab, int H, uint16_t* out,
                               unsigned* err, hipStream_t st) {
    if (n < 1 || vocab < 1 || H < 1) return hipErrorInvalidValue;
    if (H % 8 == 0 && ((uintptr_t)table & 15) == 0 && ((uintptr_t)out & 15) == 0)
        embed_gather_kernel<u32x4><<<dim3((unsigned)n), dim3(256), 0, st>>>((const u32x4*)table, ids, vocab, H / 8,
                                                                          (u32x4*)out, err);
    else
        embed_gather_kernel<uint16_t><<<dim3((unsigned)n), dim3(256), 0, st>>>(table, ids, vocab, H, out, err);
    return hipGetLastError();
}

// The k and v rows of n prompt rows (q|k|v results [n][ld], fp32) of a one-slot
// state to cache rows P .. P + n - 1 of one layer: k rotated at the row's
// position (rotate-half pairing), both rounded to the cache dtype.  One thread
// per (row, kv head, dimension).
__global__ __launch_bounds__(256) void kv_rope_append_kernel(const float* __restrict__ qkv, int ld, const int* __restrict__ pos,
                                                             const float2* __restrict__ rope, int n, int P, int Hq, int Hkv,
                                                             int D, uint16_t* __restrict__ kl, uint16_t* __restrict__ vl,
                                                             int cap, int16_t* __restrict__ table, int kv_dt) {
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= (size_t)n * Hkv * D) return;
    const int d = (int)(idx % D);
    const int g = (int)((idx / D) % Hkv);
    const int i = (int)(idx / ((size_t)D * Hkv));
    const int half = D / 2;
    const float* krow = qkv + (size_t)i * ld + (size_t)(Hq + g) * D;
    const float* vrow = qkv + (size_t)i * ld + (size_t)(Hq + Hkv + g) * D;
    const bool lo_half = d < half;
    const float xk = krow[d];
    const float xp = lo_half ? krow[d + half] : krow[d - half];
    const float2 cs = rope[(size_t)pos[i] * half + (lo_half ? d : d - half)];
    const float y = lo_half ? (xk * cs.x - xp * cs.y) : (xk * cs.x + xp * cs.y);
    const size_t off = ((size_t)g * cap + P + i) * D + d;
    kl[off] = to_half_bits(y, kv_dt);
    vl[off] = to_half_bits(vrow[d], kv_dt);
    if (table && g == 0 && d == 0) table[P + i] = 0;
}

hipError_t launch_kv_rope_append(const float* qkv, int ld, const int* pos, const float2* rope, int n, int P, int Hq, int Hkv,
                                 int D, uint16_t* kl, uint16_t* vl, int cap, int16_t* table, int kv_dt, hipStream_t st) {
    const size_t t = (size_t)n * Hkv * D;
    if (t == 0) return hipSuccess;
    kv_rope_append_kernel<<<dim3((unsigned)((t + 255) / 256)), dim3(256), 0, st>>>(qkv, ld, pos, rope, n, P, Hq, Hkv, D, kl, vl,
                                                                                    cap, table, kv_dt);
    return hipGetLastError();
}

// table[b][j] = b for j < n: every slot reads its own rows.
__global__ void table_identity_kernel(int16_t* __restrict__ table, int S, int cap, int n) {
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= (size_t)S * n) return;
    const int b = (int)(idx / n), j = (int)(idx % n);
    table[(size_t)b * cap + j] = (int16_t)b;
}

hipError_t launch_table_identity(int16_t* table, int S, int cap, int n, hipStream_t st) {
    const size_t t = (size_t)S * n;
    if (t == 0) return hipSuccess;
    table_identity_kernel<<<dim3((unsigned)((t + 255) / 256)), dim3(256), 0, st>>>(table, S, cap, n);
    return hipGetLastError();
}

}  // namespace stg
