// Persistent stage kernel: every layer of one stage forward in a single
// cooperative launch (one 256-thread workgroup per CU; one wave per SIMD, so
// each wave owns the full unified register file).
//
// Phases per layer: q|k|v GEMV -> attention -> o GEMV (+ residual) ->
// gate|up GEMV (+ SwiGLU) -> down GEMV (+ residual).  Consecutive phases are
// separated by a grid barrier built from 16 monotonically increasing 64-bit
// counters (each workgroup bumps one; wave 0 polls all of them with one
// device-coherent load per lane).  Activations cross workgroups only through
// device-coherent stores and loads, so no barrier writes back or invalidates
// the per-XCD L2s.
//
// GEMV phases: a wave owns whole weight rows (all of K), so a row's result is
// final inside the wave and no split-K exchange exists.  Lane l reads chunks
// l, l+64, ... of the row (16 bytes = 32 INT4 codes each; every wave load is
// 1 KB contiguous).  The input vector sits in LDS as fp16 pairs laid out so
// that consecutive lanes read consecutive 16 bytes.  Each wave issues the
// loads of its first weight batch of the next phase before it waits at the
// barrier, so HBM keeps streaming while the grid synchronizes, and
// double-buffers batches inside a phase.
#include "device.h"

namespace stg {

typedef unsigned long long u64;

constexpr int PS_THREADS = 256;
constexpr int PS_WAVES = PS_THREADS / 64;
static_assert(PS_WAVES == PS_WAVES_PER_WG, "host and kernel disagree on waves per workgroup");
constexpr int PS_KG = PS_THREADS / 16;       // 16-lane key groups
constexpr int PS_NC = 16;                    // barrier counters, 512 bytes apart
constexpr unsigned PS_SPIN_LIMIT = 1u << 20; // a barrier that never completes gives up (error flag)

__device__ __forceinline__ u64 load_coherent_u64(const u64* p) {
    return __hip_atomic_load(const_cast<u64*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Grid barrier number `idx` of this launch.
__device__ __forceinline__ void grid_sync(const PsArgs& a, int idx) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");   // own coherent stores have completed
    __syncthreads();
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        const unsigned n = gridDim.x;
        if (lane == 0) atomicAdd(&a.bar[(blockIdx.x % PS_NC) * 64], 1ull);
        const u64 per = (lane < PS_NC) ? (u64)((n - lane + PS_NC - 1) / PS_NC) : 0ull;
        const u64 target = (a.bar_epoch + (u64)idx + 1ull) * per;
        unsigned spins = 0;
        while (true) {
            bool ok = true;
            if (lane < PS_NC) ok = load_coherent_u64(&a.bar[lane * 64]) >= target;
            if (lane == PS_NC) ok = __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u;
            if (__all(ok)) break;
            if (!__all(lane != PS_NC || ok)) break;            // another workgroup already gave up
            __builtin_amdgcn_s_sleep(1);
            if (++spins > PS_SPIN_LIMIT) {
                if (lane == 0) atomicOr(a.err, 1u);
                break;
            }
        }
    }
    __syncthreads();
}

// ------------------------------------------------------------------ weight batches

template <int NCH>
struct WBuf {
    u32x4 w[NCH];
    uint16_t s[NCH];
};

// Rows handled by wave `gw` of `nw` in a phase with `nu` units of `RU` rows:
// units u = gw, gw + nw, ...; batch b holds units b*RB .. b*RB+RB-1 of the wave.
template <int CPL, int RB, int RU>
__device__ __forceinline__ void load_batch(WBuf<RB * RU * CPL>& B, const PsMat& W, int kc, int ng, int gchunks,
                                           int gw, int nw, int nu, int b) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < RB; ++j) {
        int u = gw + nw * (b * RB + j);
        if (u >= nu) u = nu - 1;                              // in-bounds dummy, result discarded
#pragma unroll
        for (int ru = 0; ru < RU; ++ru) {
            const size_t row = (size_t)u * RU + ru;
#pragma unroll
            for (int i = 0; i < CPL; ++i) {
                const int c = lane + 64 * i;
                B.w[(j * RU + ru) * CPL + i] = __builtin_nontemporal_load((const u32x4*)(W.w + (row * kc + c) * 16));
                B.s[(j * RU + ru) * CPL + i] = W.s[row * ng + c / gchunks];
            }
        }
    }
}

template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_rows(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROWS, 0xF, false));
}

// Wave-wide sum in a fixed order, returned as a wave-uniform value: row sums
// (DPP within 16 lanes), then row 1 += row 0 and row 3 += row 2 (row_bcast15),
// then rows 2-3 += row 1 (row_bcast31); lane 63 holds the total.
__device__ __forceinline__ float wave_sum(float v) {
    v = sum16(v);
    v += dpp_rows<0x142, 0xA>(v);
    v += dpp_rows<0x143, 0xC>(v);
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// The wave's slice of the staged input: chunk lane + 64 i of every row, as 16
// fp16 pairs per chunk.  Loaded from LDS once per phase when it fits registers.
template <int MT, int CPL>
struct XSlice {
    u32x4 q[MT][CPL][4];
};

template <int MT, int CPL>
__device__ __forceinline__ void load_xslice(XSlice<MT, CPL>& X, const uint32_t* xs, int kc, int M) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int i = 0; i < CPL; ++i)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4)
                X.q[m][i][q4] = (m < M) ? *(const u32x4*)&xs[(((size_t)m * 4 + q4) * kc + lane + 64 * i) * 4]
                                        : u32x4{0u, 0u, 0u, 0u};
}

// Dot products of one batch with the input slice (registers when XREG, else
// LDS); returns wave-uniform row sums in out[row][m].  Each 32-code chunk uses
// four independent accumulators (one per dword of codes) to keep the dot2
// chains short.
template <int MT, int CPL, int RB, int RU, bool XREG>
__device__ __forceinline__ void dot_batch(const WBuf<RB * RU * CPL>& B, const XSlice<MT, CPL>& X, const uint32_t* xs,
                                          int kc, int M, float (&out)[RB * RU][MT]) {
    const int lane = threadIdx.x & 63;
    float acc[RB * RU][MT];
#pragma unroll
    for (int r = 0; r < RB * RU; ++r)
#pragma unroll
        for (int m = 0; m < MT; ++m) acc[r][m] = 0.f;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        u32x4 xq[MT][4];
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                if constexpr (XREG) {
                    xq[m][q4] = X.q[m][i][q4];
                } else {
                    xq[m][q4] = (m < M) ? *(const u32x4*)&xs[(((size_t)m * 4 + q4) * kc + lane + 64 * i) * 4]
                                        : u32x4{0u, 0u, 0u, 0u};
                }
            }
#pragma unroll
        for (int r = 0; r < RB * RU; ++r) {
            half2_t wq[16];
            unpack_chunk(B.w[r * CPL + i], wq);
            const float sc = f16_to_f32(B.s[r * CPL + i]);
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                if (m < M) {
                    float d4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int e = 0; e < 4; ++e)
#pragma unroll
                        for (int q4 = 0; q4 < 4; ++q4) {
                            const uint32_t xe = xq[m][q4][e];
                            d4[q4] = __builtin_amdgcn_fdot2(wq[4 * q4 + e], __builtin_bit_cast(half2_t, xe), d4[q4], false);
                        }
                    acc[r][m] += sc * ((d4[0] + d4[1]) + (d4[2] + d4[3]));
                }
            }
        }
    }
#pragma unroll
    for (int r = 0; r < RB * RU; ++r)
#pragma unroll
        for (int m = 0; m < MT; ++m) out[r][m] = (m < M) ? wave_sum(acc[r][m]) : 0.f;
}

// ------------------------------------------------------------------ input staging

// Index of the uint32 holding fp16 pair p (k = 2p, 2p+1) of row m in the staged input.
__device__ __forceinline__ int xs_index(int m, int p, int kc) {
    const int c = p >> 4, pc = p & 15;
    return (((m * 4 + (pc >> 2)) * kc + c) << 2) + (pc & 3);
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Buffer resource over `bytes` bytes at p (raw dwords; out-of-range loads return 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, size_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// 16 bytes at byte offset `off`, device-coherent ("sc1": bypasses the per-XCD L2).
__device__ __forceinline__ f32x4 load4_coherent(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 16));
}

// Stage M rows of length K (a multiple of 8, padded to kc chunks with zeros)
// as fp16 pairs.  src_kind 0: fp32 rows written by other workgroups of this
// launch (coherent 16-byte loads, all issued before any is used, 8 per thread
// at a time); src_kind 1: act-dtype rows written before the launch.  With
// gamma, rows are RMS-normalized (x * rsqrt(mean(x^2) + eps) * gamma) and the
// fp32 input is also kept in xres[m][K] for the residual epilogues.
__device__ void stage_input(const void* src, int src_kind, int src_dt, int ld, int M, int K, int kc,
                            const uint16_t* gamma, int gamma_dt, float eps, uint32_t* xs, float* xres, float* red) {
    const int tid = threadIdx.x;
    const int npair = kc * 16;
    const int n4 = M * (K / 4);                      // 4-value items over all rows
    // padding pairs of every row are zero
    for (int idx = tid; idx < M * (npair - K / 2); idx += PS_THREADS) {
        const int m = idx / (npair - K / 2), p = K / 2 + idx % (npair - K / 2);
        xs[xs_index(m, p, kc)] = 0u;
    }
    auto put = [&](int it, f32x4 v) {                // item it = 4 values of row m
        const int m = it / (K / 4), k = 4 * (it % (K / 4));
        if (gamma) {
            *(f32x4*)&xres[m * K + k] = v;
        } else {
            xs[xs_index(m, k / 2, kc)] = pack_f16x2(v[0], v[1]);
            xs[xs_index(m, k / 2 + 1, kc)] = pack_f16x2(v[2], v[3]);
        }
    };
    if (src_kind == 0) {
        const __amdgpu_buffer_rsrc_t r = make_rsrc(src, (size_t)M * ld * 4);
        constexpr int B = 8;
        for (int base = 0; base < n4; base += B * PS_THREADS) {
            f32x4 v[B];
#pragma unroll
            for (int u = 0; u < B; ++u) {
                const int it = base + u * PS_THREADS + tid;
                const int m = it / (K / 4), k = 4 * (it % (K / 4));
                v[u] = load4_coherent(r, it < n4 ? (m * ld + k) * 4 : 0);
            }
#pragma unroll
            for (int u = 0; u < B; ++u) {
                const int it = base + u * PS_THREADS + tid;
                if (it < n4) put(it, v[u]);
            }
        }
    } else {
        for (int it = tid; it < n4; it += PS_THREADS) {
            const int m = it / (K / 4), k = 4 * (it % (K / 4));
            const u32x2 h = *(const u32x2*)((const uint16_t*)src + (size_t)m * ld + k);
            f32x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t w = h[e >> 1];
                v[e] = half_bits_to_f32((uint16_t)((e & 1) ? (w >> 16) : (w & 0xFFFFu)), src_dt);
            }
            put(it, v);
        }
    }
    __syncthreads();
    if (gamma) {
        for (int m = 0; m < M; ++m) {
            float ss = 0.f;
            for (int k = tid; k < K; k += PS_THREADS) ss += xres[m * K + k] * xres[m * K + k];
            red[tid] = ss;
            __syncthreads();
            for (int w = PS_THREADS / 2; w > 0; w >>= 1) {
                if (tid < w) red[tid] += red[tid + w];
                __syncthreads();
            }
            if (tid == 0) red[PS_THREADS + m] = rsqrtf(red[0] / (float)K + eps);
            __syncthreads();
        }
        for (int idx = tid; idx < M * (K / 2); idx += PS_THREADS) {
            const int m = idx / (K / 2), p = idx % (K / 2);
            const int k = 2 * p;
            const float rs = red[PS_THREADS + m];
            const uint32_t gw = *(const uint32_t*)(gamma + k);
            const float v0 = (xres[m * K + k] * rs) * half_bits_to_f32((uint16_t)(gw & 0xFFFFu), gamma_dt);
            const float v1 = (xres[m * K + k + 1] * rs) * half_bits_to_f32((uint16_t)(gw >> 16), gamma_dt);
            xs[xs_index(m, p, kc)] = pack_f16x2(v0, v1);
        }
    }
    __syncthreads();
}

// ------------------------------------------------------------------ GEMV phase

enum PsEpi : int { PE_QKV = 0, PE_RESID = 1, PE_SWIGLU = 2 };


// One GEMV phase of a workgroup.  Wave gw owns units gw, gw + nw, ... and
// streams them in batches of RB units, two batches in flight (slot 0 was
// issued before the barrier).  The streaming loop issues every load on every
// path (refills past the last batch re-read the wave's last batch) and keeps
// results in LDS, so the compiler waits for exactly the batch it consumes.
// The epilogue (residual, SwiGLU, stores) runs once per workgroup afterwards.
// res: LDS [PS_WAVES][PS_MAXU][RU][MT] floats.
template <int MT, int CPL, int RB, int RU, int EPI>
__device__ __forceinline__ void gemv_phase(const PsArgs& a, const PsMat& W, int kc, int ng, int nu,
                                           WBuf<RB * RU * CPL>& A, const uint32_t* xs, const float* xres,
                                           float* res, bool last_layer) {
    const int wave = threadIdx.x >> 6;
    const int gw = blockIdx.x * PS_WAVES + wave;
    const int nw = gridDim.x * PS_WAVES;
    const int units_w = (gw < nu) ? (nu - gw + nw - 1) / nw : 0;
    const int nb = (units_w + RB - 1) / RB;
    const int M = a.M;
    constexpr bool XREG = (MT * CPL <= 4);
    XSlice<MT, (XREG ? CPL : 1)> X;
    if constexpr (XREG) load_xslice<MT, CPL>(X, xs, kc, M);
    float* wres = res + wave * PS_MAXU * RU * MT;
    auto finish = [&](const WBuf<RB * RU * CPL>& buf, int b) {
        float v[RB * RU][MT];
        if constexpr (XREG)
            dot_batch<MT, CPL, RB, RU, true>(buf, X, xs, kc, M, v);
        else
            dot_batch<MT, CPL, RB, RU, false>(buf, *(const XSlice<MT, CPL>*)nullptr, xs, kc, M, v);
#pragma unroll
        for (int j = 0; j < RB; ++j) {
            const int lu = b * RB + j;
            if (lu < units_w) {                                  // wave-uniform; LDS only
#pragma unroll
                for (int r = 0; r < RU; ++r)
#pragma unroll
                    for (int m = 0; m < MT; ++m) wres[(lu * RU + r) * MT + m] = v[j * RU + r][m];
            }
        }
    };
    WBuf<RB * RU * CPL> B;
    load_batch<CPL, RB, RU>(B, W, kc, ng, a.gchunks, gw, nw, nu, min(1, max(nb - 1, 0)));
    for (int b0 = 0; b0 < nb; b0 += 2) {
        finish(A, b0);
        load_batch<CPL, RB, RU>(A, W, kc, ng, a.gchunks, gw, nw, nu, min(b0 + 2, max(nb - 1, 0)));
        finish(B, b0 + 1);
        load_batch<CPL, RB, RU>(B, W, kc, ng, a.gchunks, gw, nw, nu, min(b0 + 3, max(nb - 1, 0)));
    }
    __syncthreads();
    // ---- epilogue: one pass over the workgroup's results
    const int maxu = (nu + nw - 1) / nw;
    for (int idx = threadIdx.x; idx < PS_WAVES * maxu * M; idx += PS_THREADS) {
        const int w = idx / (maxu * M), lu = (idx / M) % maxu, m = idx % M;
        const int u = blockIdx.x * PS_WAVES + w + nw * lu;
        if (u >= nu) continue;
        const float* rv = res + (w * PS_MAXU + lu) * RU * MT;
        if constexpr (EPI == PE_QKV) {
            store_coherent(&a.qkv[(size_t)m * a.NQKV + u], rv[m]);
        } else if constexpr (EPI == PE_RESID) {
            const float xn = xres[m * a.H + u] + rv[m];
            store_coherent(&a.x[(size_t)m * a.H + u], xn);
            if (last_layer) ((uint16_t*)a.hidden_out)[(size_t)m * a.H + u] = to_half_bits(xn, a.act_dt);
        } else {
            const float gt = rv[m], up = rv[MT + m];
            store_coherent(&a.act[(size_t)m * a.F + u], (gt / (1.0f + expf(-gt))) * up);
        }
    }
}

// ------------------------------------------------------------------ attention phase

// One (slot, kv head, split) unit; the last split of a (slot, kv head) merges.
// Split partials are [m][h][split][D + 4] floats: max, sum, 2 pad, then D
// outputs (16-byte aligned).
template <int D, int RC>
__device__ __forceinline__ void attn_unit(const PsArgs& a, int layer, int item, int g, int split, int nsplit_of_L,
                                          float* lds) {
    constexpr int EPL = D / 16;
    constexpr int HALF = D / 2;
    constexpr int PST = D + 4;
    constexpr int KB = (RC * EPL > 32) ? 2 : 4;             // cache rows per key group per round
    const ItemDev it = a.meta.items[item];
    const ReqDev rq = a.meta.reqs[it.req];
    const int b = it.slot;
    const int P = rq.P, n = rq.n;
    const int L = P + n;
    int split_len = (L + nsplit_of_L - 1) / nsplit_of_L;
    split_len = (split_len + PS_KG - 1) / PS_KG * PS_KG;
    const int nsplit = (L + split_len - 1) / split_len;
    if (split >= nsplit) return;
    const int j0 = split * split_len, j1 = min(L, j0 + split_len);
    const int tid = threadIdx.x, kg = tid >> 4, li = tid & 15, wv = tid >> 6;
    const int Hq = a.Hq, Hkv = a.Hkv;
    const int gs = Hq / Hkv;
    const int R = gs * n;
    const int jn0 = max(j0, P);                              // this forward's rows in [jn0, j1)
    const int nn = max(0, j1 - jn0);

    float* lo = lds;                                         // [PS_WAVES][RC][D]
    float* lm = lo + PS_WAVES * RC * D;                      // [PS_WAVES][RC]
    float* ll = lm + PS_WAVES * RC;
    float* qs = ll + PS_WAVES * RC;                          // [R][D] raw q rows
    float* kn = qs + R * D;                                  // [nn][D] raw k of the new rows
    float* vn = kn + n * D;                                  // [nn][D] raw v
    uint8_t* smask = (uint8_t*)(vn + n * D);                 // [256]
    int16_t* stab = (int16_t*)(smask + 256);                 // [256]
    int* flag = (int*)(stab + 256);

    const size_t lstride = (size_t)rq.S * Hkv * rq.cap * D;
    uint16_t* kl = rq.kc + (size_t)layer * lstride;
    uint16_t* vl = rq.vc + (size_t)layer * lstride;
    const uint8_t* mask = a.meta.masks + rq.mask_off + (size_t)b * rq.mask_len;
    const int16_t* tab = rq.table + (size_t)b * rq.cap;
    const int rowbase = rq.row0 + b * n;
    const int d0 = li * EPL;
    const int jc1 = min(j1, P);

    // ---- one round of coherent 16-byte loads: q rows of this kv head group, new k and v rows
    {
        const __amdgpu_buffer_rsrc_t r = make_rsrc(a.qkv, (size_t)(rowbase + n) * a.NQKV * 4);
        const int nq4 = R * D / 4, nk4 = nn * D / 4;
        for (int x = tid; x < nq4 + 2 * nk4; x += PS_THREADS) {
            int off;
            float* dst;
            if (x < nq4) {
                const int rr = x / (D / 4), d = 4 * (x % (D / 4));
                const int i = rr / gs, h = g * gs + (rr % gs);
                off = ((rowbase + i) * a.NQKV + h * D + d) * 4;
                dst = qs + rr * D + d;
            } else {
                const int y = (x - nq4) % nk4, isv = (x - nq4) / nk4;
                const int i = (jn0 - P) + y / (D / 4), d = 4 * (y % (D / 4));
                off = ((rowbase + i) * a.NQKV + (Hq + isv * Hkv + g) * D + d) * 4;
                dst = (isv ? vn : kn) + (y / (D / 4)) * D + d;
            }
            *(f32x4*)dst = load4_coherent(r, off);
        }
    }
    __syncthreads();

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
                const int i = r / gs;
                const int pos = a.meta.positions[rowbase + i];
                qi[rr] = i;
#pragma unroll
                for (int e = 0; e < EPL; ++e) {
                    const int d = d0 + e;
                    const bool lo_half = d < HALF;
                    const float x = qs[r * D + d];
                    const float xp = qs[r * D + (lo_half ? d + HALF : d - HALF)];
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
                if (j > P + qi[rr]) continue;
                const float mn = fmaxf(mx[rr], sd);
                const float corr = exp2f(mx[rr] - mn);
                const float p = exp2f(sd - mn);
                sl[rr] = sl[rr] * corr + p;
#pragma unroll
                for (int e = 0; e < EPL; ++e) o[rr][e] = o[rr][e] * corr + p * vf[e];
                mx[rr] = mn;
            }
        };
        // cached rows through the beam table, 256 at a time
        for (int jb = j0; jb < jc1; jb += 256) {
            const int nbk = min(256, jc1 - jb);
            __syncthreads();
            for (int x = tid; x < nbk; x += PS_THREADS) {
                smask[x] = mask[jb + x];
                stab[x] = tab[jb + x];
            }
            __syncthreads();
            for (int x0 = kg; x0 < nbk; x0 += PS_KG * KB) {
                uint16_t kb[KB][EPL], vb[KB][EPL];
                bool vis[KB];
#pragma unroll
                for (int u = 0; u < KB; ++u) {
                    const int x = x0 + u * PS_KG;
                    vis[u] = (x < nbk) && smask[x] != 0;
                    if (vis[u]) {
                        const size_t off = (((size_t)stab[x] * Hkv + g) * rq.cap + (jb + x)) * D + d0;
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
                    consume(jb + x0 + u * PS_KG, kf, vf);
                }
            }
        }
        // this forward's rows: rotate k, round k and v to the cache dtype; the
        // first row pass also appends them to the cache
        for (int j = jn0 + kg; j < j1; j += PS_KG) {
            const int i = j - P;
            const int y = j - jn0;
            const int pos = a.meta.positions[rowbase + i];
            uint16_t kb[EPL], vb[EPL];
            float kf[EPL], vf[EPL];
#pragma unroll
            for (int e = 0; e < EPL; ++e) {
                const int d = d0 + e;
                const bool lo_half = d < HALF;
                const float x = kn[y * D + d];
                const float xp = kn[y * D + (lo_half ? d + HALF : d - HALF)];
                const float2 cs = a.rope[(size_t)pos * HALF + (lo_half ? d : d - HALF)];
                const float yv = lo_half ? (x * cs.x - xp * cs.y) : (x * cs.x + xp * cs.y);
                kb[e] = to_half_bits(yv, a.kv_dt);
                vb[e] = to_half_bits(vn[y * D + d], a.kv_dt);
                kf[e] = half_bits_to_f32(kb[e], a.kv_dt);
                vf[e] = half_bits_to_f32(vb[e], a.kv_dt);
            }
            if (r0 == 0) {
                const size_t off = (((size_t)b * Hkv + g) * rq.cap + j) * D + d0;
#pragma unroll
                for (int e = 0; e < EPL; ++e) {
                    kl[off + e] = kb[e];
                    vl[off + e] = vb[e];
                }
                if (layer == 0 && g == 0 && li == 0) rq.table[(size_t)b * rq.cap + j] = (int16_t)b;
            }
            if (mask[j] != 0) consume(j, kf, vf);
        }
        // merge the 4 key groups of each wave (lanes 16 apart), then the waves
#pragma unroll
        for (int rr = 0; rr < RC; ++rr) {
#pragma unroll
            for (int sh = 16; sh <= 32; sh <<= 1) {
                const float m2 = __shfl_xor(mx[rr], sh);
                const float l2 = __shfl_xor(sl[rr], sh);
                const float mn = fmaxf(mx[rr], m2);
                const float w1 = (mx[rr] == -INFINITY) ? 0.f : exp2f(mx[rr] - mn);
                const float w2 = (m2 == -INFINITY) ? 0.f : exp2f(m2 - mn);
#pragma unroll
                for (int e = 0; e < EPL; ++e) {
                    const float o2 = __shfl_xor(o[rr][e], sh);
                    o[rr][e] = o[rr][e] * w1 + o2 * w2;
                }
                sl[rr] = sl[rr] * w1 + l2 * w2;
                mx[rr] = mn;
            }
        }
        if ((tid & 63) < 16) {
#pragma unroll
            for (int rr = 0; rr < RC; ++rr) {
                if (li == 0) {
                    lm[wv * RC + rr] = mx[rr];
                    ll[wv * RC + rr] = sl[rr];
                }
#pragma unroll
                for (int e = 0; e < EPL; ++e) lo[(wv * RC + rr) * D + d0 + e] = o[rr][e];
            }
        }
        __syncthreads();
        for (int idx = tid; idx < RC * D; idx += PS_THREADS) {
            const int rr = idx / D, d = idx % D;
            const int r = r0 + rr;
            if (r >= R) continue;
            float Mx = -INFINITY;
            for (int w = 0; w < PS_WAVES; ++w) Mx = fmaxf(Mx, lm[w * RC + rr]);
            float O = 0.f, S = 0.f;
            for (int w = 0; w < PS_WAVES; ++w) {
                const float mk = lm[w * RC + rr];
                const float wt = (mk == -INFINITY) ? 0.f : exp2f(mk - Mx);
                O += lo[(w * RC + rr) * D + d] * wt;
                S += ll[w * RC + rr] * wt;
            }
            const int i = r / gs, h = g * gs + (r % gs);
            const int m = rowbase + i;
            float* pp = a.apart + (((size_t)m * Hq + h) * a.nsplit_max + split) * PST;
            store_coherent(pp + 4 + d, O);
            if (d == 0) {
                store_coherent(pp, Mx);
                store_coherent(pp + 1, S);
            }
        }
        __syncthreads();
    }

    if (!last_arrival(&a.acnt[item * Hkv + g], (unsigned)nsplit, flag)) return;
    // ---- merge the splits: weights from (max, sum) pairs, then 4 outputs per thread
    float* wgt = lo;                       // [R][nsplit]
    float* inv = wgt + R * nsplit;         // [R]
    const __amdgpu_buffer_rsrc_t pr = make_rsrc(a.apart, (size_t)MAX_ROWS * Hq * a.nsplit_max * PST * 4);
    for (int idx = tid; idx < R * nsplit; idx += PS_THREADS) {
        const int r = idx / nsplit, s2 = idx % nsplit;
        const int m = rowbase + r / gs, h = g * gs + (r % gs);
        const f32x4 ms = load4_coherent(pr, (int)(((((size_t)m * Hq + h) * a.nsplit_max + s2) * PST) * 4));
        wgt[idx] = ms[0];
        inv[R + idx] = ms[1];
    }
    __syncthreads();
    for (int r = tid; r < R; r += PS_THREADS) {
        float Mx = -INFINITY;
        for (int s2 = 0; s2 < nsplit; ++s2) Mx = fmaxf(Mx, wgt[r * nsplit + s2]);
        float S = 0.f;
        for (int s2 = 0; s2 < nsplit; ++s2) {
            const float ms = wgt[r * nsplit + s2];
            const float w = (ms == -INFINITY) ? 0.f : exp2f(ms - Mx);
            wgt[r * nsplit + s2] = w;
            S += inv[R + r * nsplit + s2] * w;
        }
        inv[r] = 1.0f / S;
    }
    __syncthreads();
    for (int idx = tid; idx < R * D / 4; idx += PS_THREADS) {
        const int r = idx / (D / 4), d = 4 * (idx % (D / 4));
        const int i = r / gs, h = g * gs + (r % gs);
        const int m = rowbase + i;
        const size_t base = (((size_t)m * Hq + h) * a.nsplit_max) * PST + 4 + d;
        f32x4 O = {0.f, 0.f, 0.f, 0.f};
        int s2 = 0;
        for (; s2 + 8 <= nsplit; s2 += 8) {
            f32x4 b8[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) b8[e] = load4_coherent(pr, (int)((base + (size_t)(s2 + e) * PST) * 4));
#pragma unroll
            for (int e = 0; e < 8; ++e) O += b8[e] * wgt[r * nsplit + s2 + e];
        }
        for (; s2 < nsplit; ++s2) O += load4_coherent(pr, (int)((base + (size_t)s2 * PST) * 4)) * wgt[r * nsplit + s2];
        float* dst = &a.o[(size_t)m * a.QD + (size_t)h * D + d];
#pragma unroll
        for (int e = 0; e < 4; ++e) store_coherent(dst + e, O[e] * inv[r]);
    }
    __syncthreads();
}

// ------------------------------------------------------------------ the kernel

// Phase-boundary timestamp (100 MHz real-time counter) for the optional trace.
__device__ __forceinline__ void stamp(const PsArgs& a, int l, int e) {
    if (a.trace && threadIdx.x == 0)
        a.trace[(size_t)blockIdx.x * a.n_layers * PS_TRACE_PER_LAYER + l * PS_TRACE_PER_LAYER + e] = wall_clock64();
}

template <int MT, int CPL_H, int CPL_Q, int CPL_F, int D, int RC>
__global__ __launch_bounds__(PS_THREADS) void stage_persistent_kernel(PsArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    float* xres = (float*)smem;                                  // [M][H] fp32 residual rows
    float* red = xres + (size_t)a.M * a.H;                       // [PS_THREADS + 16]
    float* res = red + PS_THREADS + 16;                          // [PS_WAVES][PS_MAXU][2][MT] row results
    uint32_t* xs = (uint32_t*)(res + PS_WAVES * PS_MAXU * 2 * MT);  // staged GEMV input (fp16 pairs)
    float* alds = (float*)xs;                                    // attention scratch (same space)

    // units per batch: about 8 chunks (8 KB per wave) per batch, two batches in flight
    constexpr int RB_H = (CPL_H >= 8) ? 1 : 8 / CPL_H;           // rows of K = H
    constexpr int RB_Q = (CPL_Q >= 8) ? 1 : 8 / CPL_Q;
    constexpr int RB_G = (CPL_H >= 4) ? 1 : 4 / CPL_H;           // gate|up row pairs
    constexpr int RB_F = (CPL_F >= 8) ? 1 : 8 / CPL_F;

    const int gw = blockIdx.x * PS_WAVES + (threadIdx.x >> 6);
    const int nw = gridDim.x * PS_WAVES;
    const int n_items = a.meta.n_items;
    int bar = 0;

    WBuf<RB_H * CPL_H> pq;                                       // q|k|v batch 0 of the coming layer
    load_batch<CPL_H, RB_H, 1>(pq, a.layers[0].qkv, a.kc_h, a.ng_h, a.gchunks, gw, nw, a.NQKV, 0);

    for (int l = 0; l < a.n_layers; ++l) {
        const PsLayer& Ly = a.layers[l];
        const bool last = (l == a.n_layers - 1);
        stamp(a, l, 0);
        // ---- q|k|v = RMSNorm(x) Wqkv^T
        if (l == 0)
            stage_input(a.hidden_in, 1, a.act_dt, a.H, a.M, a.H, a.kc_h, Ly.attn_norm, a.act_dt, a.eps, xs, xres, red);
        else
            stage_input(a.x, 0, DT_F32, a.H, a.M, a.H, a.kc_h, Ly.attn_norm, a.act_dt, a.eps, xs, xres, red);
        gemv_phase<MT, CPL_H, RB_H, 1, PE_QKV>(a, Ly.qkv, a.kc_h, a.ng_h, a.NQKV, pq, xs, xres, res, last);
        stamp(a, l, 1);
        grid_sync(a, bar++);
        stamp(a, l, 2);
        // ---- attention over the cache
        {
            const int units = n_items * a.Hkv * a.nsplit_max;
            for (int u = blockIdx.x; u < units; u += gridDim.x) {
                const int split = u % a.nsplit_max;
                const int ig = u / a.nsplit_max;
                attn_unit<D, RC>(a, l, ig / a.Hkv, ig % a.Hkv, split, a.nsplit_max, alds);
            }
        }
        WBuf<RB_Q * CPL_Q> po;                                   // o-projection weights stream during the barrier
        load_batch<CPL_Q, RB_Q, 1>(po, Ly.o, a.kc_q, a.ng_q, a.gchunks, gw, nw, a.H, 0);
        stamp(a, l, 3);
        grid_sync(a, bar++);
        stamp(a, l, 4);
        // ---- x += o Wo^T
        stage_input(a.o, 0, DT_F32, a.QD, a.M, a.QD, a.kc_q, nullptr, 0, 0.f, xs, nullptr, red);
        gemv_phase<MT, CPL_Q, RB_Q, 1, PE_RESID>(a, Ly.o, a.kc_q, a.ng_q, a.H, po, xs, xres, res, false);
        WBuf<RB_G * 2 * CPL_H> pg;
        load_batch<CPL_H, RB_G, 2>(pg, Ly.gu, a.kc_h, a.ng_h, a.gchunks, gw, nw, a.F, 0);
        stamp(a, l, 5);
        grid_sync(a, bar++);
        stamp(a, l, 6);
        // ---- act = silu(h2 Wg^T) * (h2 Wu^T), h2 = RMSNorm(x)
        stage_input(a.x, 0, DT_F32, a.H, a.M, a.H, a.kc_h, Ly.ffn_norm, a.act_dt, a.eps, xs, xres, red);
        gemv_phase<MT, CPL_H, RB_G, 2, PE_SWIGLU>(a, Ly.gu, a.kc_h, a.ng_h, a.F, pg, xs, xres, res, false);
        WBuf<RB_F * CPL_F> pd;
        load_batch<CPL_F, RB_F, 1>(pd, Ly.d, a.kc_f, a.ng_f, a.gchunks, gw, nw, a.H, 0);
        stamp(a, l, 7);
        grid_sync(a, bar++);
        stamp(a, l, 8);
        // ---- x += act Wd^T (the last layer also writes hidden_out)
        stage_input(a.act, 0, DT_F32, a.F, a.M, a.F, a.kc_f, nullptr, 0, 0.f, xs, nullptr, red);
        gemv_phase<MT, CPL_F, RB_F, 1, PE_RESID>(a, Ly.d, a.kc_f, a.ng_f, a.H, pd, xs, xres, res, last);
        stamp(a, l, 9);
        if (!last) {
            load_batch<CPL_H, RB_H, 1>(pq, a.layers[l + 1].qkv, a.kc_h, a.ng_h, a.gchunks, gw, nw, a.NQKV, 0);
            grid_sync(a, bar++);
        }
    }
}

template <int MT, int CPL_H, int CPL_Q, int CPL_F, int D, int RC>
hipError_t launch_ps(const PsArgs& a, int nwg, size_t lds, hipStream_t st) {
    const void* fn = (const void*)stage_persistent_kernel<MT, CPL_H, CPL_Q, CPL_F, D, RC>;
    static bool configured = false;
    if (!configured) {
        hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        configured = true;
    }
    PsArgs copy = a;
    void* args[] = {&copy};
    return hipLaunchCooperativeKernel(fn, dim3(nwg), dim3(PS_THREADS), args, (unsigned)lds, st);
}

// Shapes with a persistent instantiation: (K/2048 for K = H, Hq*D, F), head_dim,
// query rows per (slot, kv head).
bool ps_supported(int cpl_h, int cpl_q, int cpl_f, int D, int M, int rows_per_item) {
    if (M < 1 || M > PS_MAX_M) return false;
    if (cpl_h == 2 && cpl_q == 2 && cpl_f == 7 && D == 128) return rows_per_item <= 4;     // Llama-3.1-8B layers
    if (cpl_h == 4 && cpl_q == 4 && cpl_f == 14 && D == 128) return rows_per_item <= 8;    // Llama-3-70B layers
    if (cpl_h == 1 && cpl_q == 1 && cpl_f == 1 && D == 64) return rows_per_item <= 8;      // small test stages
    return false;
}

template <int MT, int CPL_H, int CPL_Q, int CPL_F, int D, int RC>
size_t ps_private_of() {
    hipFuncAttributes at{};
    if (hipFuncGetAttributes(&at, (const void*)stage_persistent_kernel<MT, CPL_H, CPL_Q, CPL_F, D, RC>) != hipSuccess) {
        (void)hipGetLastError();
        return (size_t)-1;
    }
    return at.localSizeBytes;
}

size_t ps_private_bytes(int cpl_h, int cpl_q, int cpl_f, int D, int rows_per_item) {
    if (cpl_h == 2 && cpl_q == 2 && cpl_f == 7 && D == 128) return ps_private_of<1, 2, 2, 7, 128, 4>();
    if (cpl_h == 4 && cpl_q == 4 && cpl_f == 14 && D == 128) return ps_private_of<1, 4, 4, 14, 128, 8>();
    if (cpl_h == 1 && cpl_q == 1 && cpl_f == 1 && D == 64)
        return rows_per_item <= 4 ? ps_private_of<1, 1, 1, 1, 64, 4>() : ps_private_of<1, 1, 1, 1, 64, 8>();
    return (size_t)-1;
}

hipError_t launch_persistent(const PsArgs& a, int cpl_h, int cpl_q, int cpl_f, int D, int rows_per_item, int nwg,
                             size_t lds, hipStream_t st) {
    if (!ps_supported(cpl_h, cpl_q, cpl_f, D, a.M, rows_per_item)) return hipErrorInvalidValue;
    if (cpl_h == 2 && cpl_q == 2 && cpl_f == 7 && D == 128) return launch_ps<1, 2, 2, 7, 128, 4>(a, nwg, lds, st);
    if (cpl_h == 4 && cpl_q == 4 && cpl_f == 14 && D == 128) return launch_ps<1, 4, 4, 14, 128, 8>(a, nwg, lds, st);
    if (cpl_h == 1 && cpl_q == 1 && cpl_f == 1 && D == 64)
        return rows_per_item <= 4 ? launch_ps<1, 1, 1, 1, 64, 4>(a, nwg, lds, st) : launch_ps<1, 1, 1, 1, 64, 8>(a, nwg, lds, st);
    return hipErrorInvalidValue;
}

// Largest dynamic LDS any instantiation asks for at this shape and row count.
size_t ps_lds_bytes(int H, int QD, int F, int kc_h, int kc_q, int kc_f, int D, int M) {
    (void)QD; (void)F;
    const int kcmax = kc_h > kc_q ? (kc_h > kc_f ? kc_h : kc_f) : (kc_q > kc_f ? kc_q : kc_f);
    const size_t xs = (size_t)M * kcmax * 64;                                // fp16 pairs
    const size_t att = (size_t)PS_WAVES * 8 * D * 4 + 2 * PS_WAVES * 8 * 4 + (8 + 2 * M) * D * 4 + 768 + 16;
    const size_t head = (size_t)M * H * 4 + (PS_THREADS + 16) * 4 + (size_t)PS_WAVES * PS_MAXU * 2 * M * 4;
    return head + (xs > att ? xs : att);
}

// Row-layout repack: dest row = row_off + r (map 0), 2r (map 1, gate), 2r + 1 (map 2, up).
__global__ void repack_rows_kernel(const uint8_t* __restrict__ q, const uint16_t* __restrict__ s, int n, int k, int g,
                                   uint8_t* __restrict__ w_out, uint16_t* __restrict__ s_out, int kc, int ng,
                                   int row_off, int row_map) {
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= (size_t)n * kc) return;
    const int r = (int)(idx / kc), c = (int)(idx % kc);
    const int kb = (k + 1) / 2;
    const int dr = row_map == 0 ? row_off + r : 2 * r + (row_map == 2 ? 1 : 0);
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
    *(u32x4*)(w_out + ((size_t)dr * kc + c) * 16) = o;
    const int ngs = (k + g - 1) / g;
    if ((c * 32) % g == 0 && c * 32 / g < ngs) s_out[(size_t)dr * ng + c * 32 / g] = s[(size_t)r * ngs + c * 32 / g];
}

hipError_t launch_repack_rows(const uint8_t* q, const uint16_t* s, int n, int k, int g, uint8_t* w_out, uint16_t* s_out,
                              int kc, int ng, int row_off, int row_map, hipStream_t st) {
    const size_t nc = (size_t)n * kc;
    repack_rows_kernel<<<dim3((unsigned)((nc + 255) / 256)), dim3(256), 0, st>>>(q, s, n, k, g, w_out, s_out, kc, ng,
                                                                                row_off, row_map);
    return hipGetLastError();
}

__global__ void dequant_rows_kernel(PsMat m, int kc, int ng, int gchunks, int k, int row_off, int row_map, int n_rows,
                                    float* __restrict__ out) {
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= (size_t)n_rows * kc) return;
    const int r = (int)(idx / kc), c = (int)(idx % kc);
    const int dr = row_map == 0 ? row_off + r : 2 * r + (row_map == 2 ? 1 : 0);
    const u32x4 w = *(const u32x4*)(m.w + ((size_t)dr * kc + c) * 16);
    half2_t h[16];
    unpack_chunk(w, h);
    const float sc = f16_to_f32(m.s[(size_t)dr * ng + c / gchunks]);
#pragma unroll
    for (int p = 0; p < 16; ++p)
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int kk = c * 32 + 2 * p + e;
            if (kk < k) out[(size_t)r * k + kk] = (float)h[p][e] * sc;
        }
}

hipError_t launch_dequant_rows(const PsMat& m, int kc, int ng, int gchunks, int k, int row_off, int row_map, int n_rows,
                               float* out, hipStream_t st) {
    const size_t nc = (size_t)n_rows * kc;
    dequant_rows_kernel<<<dim3((unsigned)((nc + 255) / 256)), dim3(256), 0, st>>>(m, kc, ng, gchunks, k, row_off, row_map,
                                                                                  n_rows, out);
    return hipGetLastError();
}

}  // namespace stg
