// Single-launch stage forward for one decode row (the "stream kernel").
//
// One workgroup per CU, made of SK_CW compute waves and one control wave; all
// workgroups are resident at once (checked when the stage is created) and hand
// values to each other only through flag words (a value and the number of the
// exchange it belongs to in one store), never through a grid barrier.
//
// Compute waves read every weight and cache byte the step needs exactly once,
// in one fixed order per wave: for each layer, the wave's q|k|v weight rows,
// its cache rows (K, V) of the layer's attention, then its o, gate|up and down
// weight rows.  Each wave keeps S direct-to-LDS loads (global_load_lds_dwordx4,
// 1 KB per wave) in flight in a private LDS ring and refills a slot as soon as
// it has consumed it, so the stream runs ahead across phase and layer
// boundaries while the exchanges complete.  Compute waves also poll the
// exchanged inputs (attention output, residual, SwiGLU output) into LDS; they
// synchronize with the control wave through s_barrier only and read LDS
// through inline ds_read with explicit waits (the compiler does not track
// direct-to-LDS loads).
//
// The control wave does the work on the critical path between phases: the
// epilogues (rotary embedding, residual, SwiGLU), publishing each phase's
// outputs as flag words, the q|k|v and split-partial waits, the next phase's
// scale rows and norm weights, and the split-KV merge.
//
// GEMV phases: a wave owns whole weight rows (all of K); lane l multiplies
// chunks l, l + 64, ... (32 codes each) with its slice of the input, which it
// keeps in registers for the whole phase.  The down projection (K = SK_CW
// blocks of 2048) is split by column block instead: wave c takes block c of
// every row of the workgroup.  Attention: workgroup w < Hkv * nsplit owns kv
// head w / nsplit and one contiguous split of the cached rows; each compute
// wave reduces its share of the split to an online-softmax partial, the
// control wave merges the waves (and this forward's own new row) and publishes
// the split's partial, and every split's workgroup then merges one slice of
// the head's outputs over all splits.
//
// A wait that does not complete within a.spin_limit polling passes gives up:
// it sets the stage's error flag, every later wait of the launch polls once,
// and the launch finishes with invalid outputs that the host reports.
#include "device.h"

namespace stg {

typedef unsigned long long u64;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int SK_THREADS = (SK_CW + 1) * 64;

// ------------------------------------------------------------------ LDS by address, explicit waits

__device__ __forceinline__ void vm_wait_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
template <int N>
__device__ __forceinline__ void vm_wait() {
    static_assert(N >= 0 && N <= 63, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void lgkm_wait_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// Workgroup barrier that does not wait for outstanding global loads.
__device__ __forceinline__ void wg_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ u32x4 lds_rd16(uint32_t a) {
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a));
    return v;
}
__device__ __forceinline__ u32x2 lds_rd8(uint32_t a) {
    u32x2 v;
    asm volatile("ds_read_b64 %0, %1" : "=v"(v) : "v"(a));
    return v;
}
__device__ __forceinline__ uint32_t lds_rdu16(uint32_t a) {
    uint32_t v;
    asm volatile("ds_read_u16 %0, %1" : "=v"(v) : "v"(a));
    return v;
}
__device__ __forceinline__ void lds_wr4(uint32_t a, float v) {
    asm volatile("ds_write_b32 %0, %1" ::"v"(a), "v"(v) : "memory");
}
__device__ __forceinline__ void lds_wr16(uint32_t a, f32x4 v) {
    asm volatile("ds_write_b128 %0, %1" ::"v"(a), "v"(v) : "memory");
}
// After lgkm_wait_all: makes `v` depend on the wait, so no use moves above it.
__device__ __forceinline__ void touch(u32x4& v) { asm volatile("" : "+v"(v)); }
__device__ __forceinline__ void touch(uint32_t& v) { asm volatile("" : "+v"(v)); }
__device__ __forceinline__ void touch(u32x2& v) { asm volatile("" : "+v"(v)); }

// (x & m) | c for c free of m's bits, in one instruction (mask from an SGPR,
// constant from a VGPR: a VOP3 encoding takes no literal operands).
__device__ __forceinline__ uint32_t bfi(uint32_t m, uint32_t x, uint32_t c) {
    uint32_t r;
    asm volatile("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "s"(m), "v"(x), "v"(c));
    return r;
}

// Direct-to-LDS load: lane l's 16 bytes at g land at LDS byte lds + 16 l (lds is wave-uniform).
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
    __builtin_amdgcn_global_load_lds(g, (lds_ptr_t)(uintptr_t)lds, 16, 0, 2 /* nt: streamed once */);
}


__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }

// ------------------------------------------------------------------ device-coherent exchange

__device__ __forceinline__ u64 load_coherent_u64(const u64* p) {
    return __hip_atomic_load(const_cast<u64*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_coherent_u32(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, size_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
// 16 bytes at byte offset `off`, device-coherent ("sc1": bypasses the per-XCD L2).
__device__ __forceinline__ f32x4 load4_coherent(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 16));
}

template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_rows(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROWS, 0xF, false));
}
// Wave-wide sum in a fixed order, returned as a wave-uniform value.
__device__ __forceinline__ float wave_sum(float v) {
    v = sum16(v);
    v += dpp_rows<0x142, 0xA>(v);     // row_bcast15: rows 1, 3 += rows 0, 2
    v += dpp_rows<0x143, 0xC>(v);     // row_bcast31: rows 2, 3 += row 1
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}
// Sum over aligned groups of N lanes (8 or 16); every lane of a group receives it.
template <int N>
__device__ __forceinline__ float group_sum(float v) {
    static_assert(N == 8 || N == 16, "group size");
    v += dpp_f<0xB1>(v);
    v += dpp_f<0x4E>(v);
    v += dpp_f<0x141>(v);             // row_half_mirror: sums of 8
    if constexpr (N == 16) v += dpp_f<0x140>(v);
    return v;
}

// The values of v in this lane and in lane ^ sh.  For sh = 16 and 32 one swap
// instruction returns, in every lane, the value of the lower and of the upper
// lane of the pair (a = lower, b = upper); otherwise a is this lane's value.
__device__ __forceinline__ void lane_pair(float v, int sh, float& a, float& b) {
    const uint32_t u = __float_as_uint(v);
    if (sh == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
        a = __uint_as_float(r[0]);
        b = __uint_as_float(r[1]);
    } else if (sh == 32) {
        const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
        a = __uint_as_float(r[0]);
        b = __uint_as_float(r[1]);
    } else {
        a = v;
        b = __shfl_xor(v, sh);
    }
}

// Sums of four rows' per-lane partials v0..v3 at once, in a fixed order:
// lane l < 4 receives the sum of v_l over the wave.  Each step halves the
// values per lane by exchanging the one the partner keeps (xor 1, xor 2), then
// the 16-lane rows and the four rows of the wave are added.
__device__ __forceinline__ float sum4_rows(float v0, float v1, float v2, float v3, int lane) {
    const bool b0 = (lane & 1) != 0, b1 = (lane & 2) != 0;
    float k0 = b0 ? v1 : v0;
    k0 += dpp_f<0xB1>(b0 ? v0 : v1);  // quad_perm [1,0,3,2]: lane ^ 1
    float k1 = b0 ? v3 : v2;
    k1 += dpp_f<0xB1>(b0 ? v2 : v3);
    float k = b1 ? k1 : k0;
    k += dpp_f<0x4E>(b1 ? k0 : k1);   // quad_perm [2,3,0,1]: lane ^ 2; lane holds row lane & 3
    k += dpp_f<0x124>(k);             // row_ror:4
    k += dpp_f<0x128>(k);             // row_ror:8: the 16-lane row
    float lo, hi;
    lane_pair(k, 16, lo, hi);
    k = lo + hi;
    lane_pair(k, 32, lo, hi);
    return lo + hi;
}

// ------------------------------------------------------------------ flag-in-data exchange
//
// A 32-bit value exchanged between workgroups travels in one 8-byte word with
// the number of the write that produced it in the high half, written with one
// device-coherent 8-byte store.  A reader polls the words it needs until each
// carries the expected number: no acknowledgement, counter or barrier sits
// between producer and consumer.  A buffer is only rewritten (with a higher
// number) after every reader of its previous contents has finished with it,
// which the data dependencies of the forward guarantee (see control_main).

__device__ __forceinline__ void ll_store(u64* p, uint32_t v, uint32_t flag) {
    __hip_atomic_store(p, ((u64)flag << 32) | (u64)v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Two adjacent flag words (16-byte aligned, byte offset off in the buffer
// behind r) in one device-coherent 16-byte store: each 8-byte half carries the
// write number, and readers check both halves.  Fewer store instructions before
// a wave's next poll: its loads wait for its stores' acknowledgement.
__device__ __forceinline__ void ll_store2(__amdgpu_buffer_rsrc_t r, int off, uint32_t v0, uint32_t v1, uint32_t flag) {
    __builtin_amdgcn_raw_buffer_store_b128(u32x4{v0, flag, v1, flag}, r, off, 0, 16);
}
// A 16-bit value with the low 16 bits of the write number in one 4-byte word.
// Every buffer is rewritten at each use, so a stale word carries a number at
// most a few hundred writes old, never equal to the expected one modulo 2^16.
__device__ __forceinline__ void ll_store16(uint32_t* p, uint16_t v, uint32_t flag) {
    __hip_atomic_store(p, (uint32_t)v | (flag << 16), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The lane index, recomputed where it is called: offsets derived from it are
// then not hoisted out of the layer loop (where they would stay live throughout).
__device__ __forceinline__ int fresh_lane() {
    int l = threadIdx.x & 63;
    asm volatile("" : "+v"(l));
    return l;
}

// Polls NP 16-byte pieces of the buffer behind r, piece i at byte offset off[i]
// and wanted when bit i of `use` is set, until every word of every wanted piece
// carries `flag` (pieces i < N16 hold four 4-byte words, the others two 8-byte
// words); take(i, piece) receives each piece once, as
// soon as it is complete.  Every pass issues all its loads at once: a piece
// already taken gets an offset past the end of the buffer, which the hardware
// answers with zeros without a memory access.  Returns false when the wait
// gives up (error flag set) or once any workgroup has given up; with ok false
// it makes one pass and does not wait.
// With tracing on, wait number tw (0..5) of layer tl records its passes and end time.
template <int NP, int N16 = 0, class Take>
__device__ __forceinline__ bool ll_wait(const PsArgs& a, __amdgpu_buffer_rsrc_t r, const int (&off)[NP], uint32_t use,
                                        uint32_t flag, Take&& take, bool ok, int tl = -1, int tw = -1) {
    static_assert(NP <= 32, "one bit per piece");
    constexpr int OOB = 0x7FFFFFF0;
    const int lane = threadIdx.x & 63;
    uint32_t pend = use;
    unsigned spins = 0;
    const u64 t_issue = (a.trace && tw >= 0) ? wall_clock64() : 0ull;   // stored at the end: a store now would
    while (true) {                                                      // join this wave's load count
        u32x4 v[NP];
#pragma unroll
        for (int i = 0; i < NP; ++i)
            v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, ((pend >> i) & 1u) ? off[i] : OOB, 0, 16));
        uint32_t bad = 0u;
        if (lane == 0) bad = __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int i = 0; i < NP; ++i) {
            bool rd;
            if (i < N16) {
                const uint32_t w0 = v[i][0], w1 = v[i][1], w2 = v[i][2], w3 = v[i][3];
                const uint32_t f16 = flag & 0xFFFFu;
                rd = (w0 >> 16) == f16 && (w1 >> 16) == f16 && (w2 >> 16) == f16 && (w3 >> 16) == f16;
            } else {
                const uint32_t f0 = v[i][1], f1 = v[i][3];
                rd = f0 == flag && f1 == flag;
            }
            if (((pend >> i) & 1u) && rd) {
                take(i, v[i]);
                pend &= ~(1u << i);
            }
        }
        if (a.trace && tw >= 0 && lane == 0 && spins == 0)
            a.trace[((size_t)blockIdx.x * a.n_layers + tl) * PS_TRACE_PER_LAYER + 28 + (tw == 3 ? 0 : tw == 5 ? 1 : 2)] = wall_clock64();
        if (__all(pend == 0u)) {
            if (a.trace && tw >= 0 && lane == 0) {
                u64* tr = a.trace + ((size_t)blockIdx.x * a.n_layers + tl) * PS_TRACE_PER_LAYER;
                tr[16 + tw] = spins + 1;
                tr[22 + tw] = wall_clock64();
                tr[32 + tw] = t_issue;
            }
            return ok;
        }
        if (!ok) return false;
        if (__any(bad != 0u)) return false;                // another workgroup already gave up
        if (++spins > a.spin_limit) {
            if (lane == 0) atomicOr(a.err, 1u);
            return false;
        }
    }
}

// Compute wave 0 keeps its stamps in LDS (a global store would join its load count).
__device__ __forceinline__ void cstamp(const PsArgs& a, uint32_t dbg, int k) {
    if (a.trace && threadIdx.x == 0) {
        const u64 t = wall_clock64();
        asm volatile("ds_write_b64 %0, %1" ::"v"(dbg + 8 * k), "v"(t) : "memory");
    }
}

__device__ __forceinline__ void stamp(const PsArgs& a, int l, int e) {
    if (a.trace && (threadIdx.x & 63) == 0)
        a.trace[(size_t)blockIdx.x * a.n_layers * PS_TRACE_PER_LAYER + l * PS_TRACE_PER_LAYER + e] = wall_clock64();
}

// ------------------------------------------------------------------ row partition

// Rows [first, first + count) of an N-row matrix owned by workgroup w (rpw
// rows each) and, within it, by compute wave cw.
struct Rows {
    int first, count, local;   // local: index of `first` within the workgroup's rows
};
__device__ __forceinline__ Rows wave_rows(int N, int rpw, int w, int cw) {
    const int rpc = (rpw + SK_CW - 1) / SK_CW;
    const int wg0 = w * rpw;
    const int wg1 = min(N, wg0 + rpw);
    const int a0 = min(wg1, wg0 + cw * rpc);
    const int a1 = min(wg1, a0 + rpc);
    return Rows{a0, max(0, a1 - a0), a0 - wg0};
}

// ------------------------------------------------------------------ compute waves

// Attention split geometry shared by both roles.
template <int D>
struct AttGeo {
    static constexpr int LPR = D / 8;         // lanes per cache row (16 bytes each)
    static constexpr int RPS = 64 / LPR;      // cache rows per slot
};

// Position bookkeeping of one compute wave's ring: p is the stream position
// of the next slot to consume, ri its ring index; loads are issued strictly in
// stream order, S positions ahead, so before consuming position q (with the
// refill of q - 1 issued) exactly S - 1 younger loads may be in flight while
// q <= pmax, and fewer near the end of the stream.
struct Ring {
    uint32_t base;            // LDS byte address of slot 0 (lane i's 16 bytes of a slot at 16 i)
    int p, ri, pmax;
    __device__ __forceinline__ uint32_t addr(int r) const { return base + (uint32_t)r * SK_SLOT; }
    __device__ __forceinline__ static int next(int r, int S) { return r + 1 == S ? 0 : r + 1; }
};

// One GEMV segment: `nrows` rows (whole K each) from the ring, results to LDS res.
//
// INT4 decode: a dword of codes holds k..k+7; masking with 0x000F000F /
// 0x00F000F0 (of x and x >> 8) and or-ing 0x6400 gives fp16 pairs equal to
// 1024 + u (pairs (k, k+1), (k+4, k+5)) or 1024 + 16u (pairs (k+2, k+3),
// (k+6, k+7)) with u = q + 8.  The input slice is prepared once per segment:
// the values that meet a 1024 + 16u code are divided by 16 (exact: a power of
// two), so every product of a chunk adds into one sum, which starts from the
// chunk's correction -(1032 S_lo + 72 S_hi) (S_lo, S_hi: the chunk's input
// sums over the two kinds of position); then sum q x is the sum itself.
//
// Rows are consumed whole, four at a time (one wave-wide reduction per four
// rows), from two register sets used alternately: while row r computes from
// one set, the codes and scales of row r + 1 are read into the other.
template <int S, class Issue>
__device__ __forceinline__ void gemv_seg1(const PsArgs& a, Issue& issue, Ring& rg, int nrows, int rlocal, int ng,
                                          uint32_t sb, uint32_t xs, uint32_t res);

template <int CPL, int S, class Issue>
__device__ __forceinline__ void gemv_seg(const PsArgs& a, Issue& issue, Ring& rg, int nrows, int rlocal, int ng,
                                         uint32_t sb, uint32_t xs, uint32_t res) {
    static_assert(S >= 2 * CPL, "the ring must hold two rows");
    static_assert(CPL <= 4, "the input slice is kept in registers");
    if constexpr (CPL == 1) {
        gemv_seg1<S>(a, issue, rg, nrows, rlocal, ng, sb, xs, res);
        return;
    }
    if (nrows == 0) return;
    const int lane = threadIdx.x & 63;
    const half2_t one2 = {(_Float16)1.0f, (_Float16)1.0f};
    const half2_t sixteenth2 = {(_Float16)0.0625f, (_Float16)0.0625f};
    // chunk lane + 64 i of the input as 16 fp16 pairs (prepared), and its correction
    const uint32_t xl = xs + 64 * lane;                      // chunk `lane`; chunk lane + 64 i is 4 KB i further
    u32x4 xq[CPL][4];
    float ncorr[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) xq[i][q4] = lds_rd16(xl + 4096 * i + 16 * q4);
    lgkm_wait_all();
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        float slo = 0.f, shi = 0.f;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            touch(xq[i][q4]);
            // elements are taken into scalars before any bit cast
            const uint32_t e0 = xq[i][q4][0], e1 = xq[i][q4][1], e2 = xq[i][q4][2], e3 = xq[i][q4][3];
            slo = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, e0), one2, slo, false);
            slo = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, e2), one2, slo, false);
            shi = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, e1), one2, shi, false);
            shi = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, e3), one2, shi, false);
            const half2_t h1 = __builtin_bit_cast(half2_t, e1) * sixteenth2;
            const half2_t h3 = __builtin_bit_cast(half2_t, e3) * sixteenth2;
            xq[i][q4] = u32x4{e0, __builtin_bit_cast(uint32_t, h1), e2, __builtin_bit_cast(uint32_t, h3)};
        }
        ncorr[i] = -(1032.0f * slo + 72.0f * shi);
        asm volatile("" : "+v"(ncorr[i]));                  // computed here, not inside the row loop
    }
    const int gstep = 128 / a.gchunks;                      // scale bytes between chunk i and i + 1 of a row
    const uint32_t sl = sb + 2 * (uint32_t)(lane / a.gchunks) + 2 * rlocal * ng;
    const uint32_t lane16 = 16 * lane;
    uint32_t magic = 0x64006400u;
    asm volatile("" : "+v"(magic));                         // kept in a VGPR for v_bfi

    u32x4 w0[CPL], w1[CPL];
    uint32_t c0[CPL], c1[CPL];
    auto read_row = [&](int r, u32x4 (&w)[CPL], uint32_t (&sc)[CPL]) {
        int ri = rg.ri;
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
            w[i] = lds_rd16(rg.addr(ri) + lane16);
            sc[i] = lds_rdu16(sl + 2 * r * ng + gstep * i);
            ri = Ring::next(ri, S);
        }
    };
    // Row r from (cw, cs): its slots are refilled (they are in registers), the
    // next row is read into (nw, ns) (after the last row the reads fall on a
    // ring slot and a scale of this segment, valid LDS addresses, and are not
    // used), and the row's per-lane partial is returned once those reads are done.
    auto row = [&](int r, const u32x4 (&cw)[CPL], const uint32_t (&cs)[CPL], u32x4 (&nw)[CPL],
                   uint32_t (&ns)[CPL]) -> float {
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
            issue(rg.addr(rg.ri));
            rg.ri = Ring::next(rg.ri, S);
        }
        rg.p += CPL;
        if (r + 1 < nrows) {
            // younger than the next row's last slot: S - CPL while the stream is not near its end
            if (rg.p <= rg.pmax) vm_wait<S - CPL>(); else vm_wait_all();
        }
        read_row(min(r + 1, nrows - 1), nw, ns);
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
            float t0 = ncorr[i], t1 = 0.f;
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const uint32_t x = cw[i][q4];
                const uint32_t y = x >> 8;
                const uint32_t p0 = bfi(0x000F000Fu, x, magic);
                const uint32_t p1 = bfi(0x00F000F0u, x, magic);
                const uint32_t p2 = bfi(0x000F000Fu, y, magic);
                const uint32_t p3 = bfi(0x00F000F0u, y, magic);
                const uint32_t x0 = xq[i][q4][0], x1 = xq[i][q4][1], x2 = xq[i][q4][2], x3 = xq[i][q4][3];
                t0 = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p0), __builtin_bit_cast(half2_t, x0), t0, false);
                t1 = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p1), __builtin_bit_cast(half2_t, x1), t1, false);
                t0 = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p2), __builtin_bit_cast(half2_t, x2), t0, false);
                t1 = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p3), __builtin_bit_cast(half2_t, x3), t1, false);
            }
            acc = __builtin_fmaf(f16_to_f32((uint16_t)cs[i]), t0 + t1, acc);
        }
        // the wait takes acc as an operand, so this row's arithmetic is issued before it
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(acc)::"memory");
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
            touch(nw[i]);
            touch(ns[i]);
        }
        return acc;
    };
    if (rg.p <= rg.pmax) vm_wait<S - CPL>(); else vm_wait_all();   // S + p <= total: S - CPL younger loads
    read_row(0, w0, c0);
    lgkm_wait_all();
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        touch(w0[i]);
        touch(c0[i]);
    }
    int r = 0;
    for (; r + 4 <= nrows; r += 4) {
        const float a0 = row(r, w0, c0, w1, c1);
        const float a1 = row(r + 1, w1, c1, w0, c0);
        const float a2 = row(r + 2, w0, c0, w1, c1);
        const float a3 = row(r + 3, w1, c1, w0, c0);
        const float rs = sum4_rows(a0, a1, a2, a3, lane);
        if (lane < 4) lds_wr4(res + 4 * (rlocal + r + lane), rs);
    }
    if (r < nrows) {                                        // one to three rows left
        const int nt = nrows - r;
        const float a0 = row(r, w0, c0, w1, c1);
        float a1 = 0.f, a2 = 0.f;
        if (nt > 1) a1 = row(r + 1, w1, c1, w0, c0);
        if (nt > 2) a2 = row(r + 2, w0, c0, w1, c1);
        const float rs = sum4_rows(a0, a1, a2, 0.f, lane);
        if (lane < nt) lds_wr4(res + 4 * (rlocal + r + lane), rs);
    }
}

// The one-chunk form of gemv_seg (rows of K = 2048, one slot each): every row
// multiplies the same input chunk, so rows go two at a time; a step holds the
// arithmetic of two slots, which covers the LDS reads of the next step's two
// slots and scales (one slot of arithmetic does not).
template <int S, class Issue>
__device__ __forceinline__ void gemv_seg1(const PsArgs& a, Issue& issue, Ring& rg, int nrows, int rlocal, int ng,
                                          uint32_t sb, uint32_t xs, uint32_t res) {
    static_assert(S >= 4, "the ring must hold two steps");
    if (nrows == 0) return;
    const int lane = threadIdx.x & 63;
    const half2_t one2 = {(_Float16)1.0f, (_Float16)1.0f};
    const half2_t sixteenth2 = {(_Float16)0.0625f, (_Float16)0.0625f};
    u32x4 xq[4];
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) xq[q4] = lds_rd16(xs + 64 * lane + 16 * q4);
    lgkm_wait_all();
    float ncorr;
    {
        float slo = 0.f, shi = 0.f;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            touch(xq[q4]);
            const uint32_t e0 = xq[q4][0], e1 = xq[q4][1], e2 = xq[q4][2], e3 = xq[q4][3];
            slo = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, e0), one2, slo, false);
            slo = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, e2), one2, slo, false);
            shi = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, e1), one2, shi, false);
            shi = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, e3), one2, shi, false);
            const half2_t h1 = __builtin_bit_cast(half2_t, e1) * sixteenth2;
            const half2_t h3 = __builtin_bit_cast(half2_t, e3) * sixteenth2;
            xq[q4] = u32x4{e0, __builtin_bit_cast(uint32_t, h1), e2, __builtin_bit_cast(uint32_t, h3)};
        }
        ncorr = -(1032.0f * slo + 72.0f * shi);
        asm volatile("" : "+v"(ncorr));
    }
    const uint32_t sl = sb + 2 * (uint32_t)(lane / a.gchunks) + 2 * rlocal * ng;
    const uint32_t lane16 = 16 * lane;
    uint32_t magic = 0x64006400u;
    asm volatile("" : "+v"(magic));

    u32x4 w0[2], w1[2];
    uint32_t c0[2], c1[2];
    // rows r, r + 1 (a row past the segment reads the next ring slot and the
    // segment's last scale: valid LDS addresses, not used)
    auto read_pair = [&](int r, u32x4 (&w)[2], uint32_t (&sc)[2]) {
        const int r1 = Ring::next(rg.ri, S);
        w[0] = lds_rd16(rg.addr(rg.ri) + lane16);
        w[1] = lds_rd16(rg.addr(r1) + lane16);
        sc[0] = lds_rdu16(sl + 2 * min(r, nrows - 1) * ng);
        sc[1] = lds_rdu16(sl + 2 * min(r + 1, nrows - 1) * ng);
    };
    auto dot = [&](const u32x4& cw, uint32_t cs) -> float {
        float t0 = ncorr, t1 = 0.f;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            const uint32_t x = cw[q4];
            const uint32_t y = x >> 8;
            const uint32_t p0 = bfi(0x000F000Fu, x, magic);
            const uint32_t p1 = bfi(0x00F000F0u, x, magic);
            const uint32_t p2 = bfi(0x000F000Fu, y, magic);
            const uint32_t p3 = bfi(0x00F000F0u, y, magic);
            const uint32_t x0 = xq[q4][0], x1 = xq[q4][1], x2 = xq[q4][2], x3 = xq[q4][3];
            t0 = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p0), __builtin_bit_cast(half2_t, x0), t0, false);
            t1 = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p1), __builtin_bit_cast(half2_t, x1), t1, false);
            t0 = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p2), __builtin_bit_cast(half2_t, x2), t0, false);
            t1 = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p3), __builtin_bit_cast(half2_t, x3), t1, false);
        }
        return f16_to_f32((uint16_t)cs) * (t0 + t1);
    };
    // Rows r, r + 1 (only r when it is the last) from (cw, cs): their slots are
    // refilled, the next step is read into (nw, ns), and the rows' per-lane
    // partials are returned once those reads are done.
    auto step = [&](int r, const u32x4 (&cw)[2], const uint32_t (&cs)[2], u32x4 (&nw)[2], uint32_t (&ns)[2],
                    float& p0, float& p1) {
        const bool two = r + 1 < nrows;                     // wave-uniform
        issue(rg.addr(rg.ri));
        rg.ri = Ring::next(rg.ri, S);
        if (two) {
            issue(rg.addr(rg.ri));
            rg.ri = Ring::next(rg.ri, S);
        }
        rg.p += two ? 2 : 1;
        if (r + 2 < nrows) {
            // the next step's two positions: S - 2 younger loads while the stream is not near its end
            if (rg.p + 1 <= rg.pmax) vm_wait<S - 2>(); else vm_wait_all();
        }
        read_pair(r + 2, nw, ns);
        p0 = dot(cw[0], cs[0]);
        p1 = two ? dot(cw[1], cs[1]) : 0.f;
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(p0), "+v"(p1)::"memory");
        touch(nw[0]);
        touch(nw[1]);
        touch(ns[0]);
        touch(ns[1]);
    };
    if (rg.p + 1 <= rg.pmax) vm_wait<S - 2>(); else vm_wait_all();
    read_pair(0, w0, c0);
    lgkm_wait_all();
    touch(w0[0]);
    touch(w0[1]);
    touch(c0[0]);
    touch(c0[1]);
    int r = 0;
    for (; r + 4 <= nrows; r += 4) {
        float a0, a1, a2, a3;
        step(r, w0, c0, w1, c1, a0, a1);
        step(r + 2, w1, c1, w0, c0, a2, a3);
        const float rs = sum4_rows(a0, a1, a2, a3, lane);
        if (lane < 4) lds_wr4(res + 4 * (rlocal + r + lane), rs);
    }
    if (r < nrows) {                                        // one to three rows left
        const int nt = nrows - r;
        float a0, a1, a2 = 0.f, a3 = 0.f;
        step(r, w0, c0, w1, c1, a0, a1);
        if (nt > 2) step(r + 2, w1, c1, w0, c0, a2, a3);
        const float rs = sum4_rows(a0, a1, a2, a3, lane);
        if (lane < nt) lds_wr4(res + 4 * (rlocal + r + lane), rs);
    }
}

// Slot range of one wave in a long-row GEMV segment (input chunks read from
// LDS): the workgroup's rows x CPL chunks are split evenly over its compute
// waves in row-major order, so a row may be shared by two waves.  Partials go
// to res[2 r] (the part holding the row's first chunk) and res[2 r + 1].
__host__ __device__ __forceinline__ int kslot_per_wave(int rows, int cpl) { return (rows * cpl + SK_CW - 1) / SK_CW; }

template <int CPL, int S, class Issue>
__device__ __forceinline__ void gemv_seg_k(const PsArgs& a, Issue& issue, Ring& rg, int s0, int ns, int ng, uint32_t sb,
                                           uint32_t xs, uint32_t res) {
    if (ns == 0) return;
    const int lane = threadIdx.x & 63;
    const half2_t one2 = {(_Float16)1.0f, (_Float16)1.0f};
    const uint32_t xl = xs + 64 * lane;                      // chunk `lane`; chunk lane + 64 i is 4 KB i further
    const int gstep = 128 / a.gchunks;
    const uint32_t sl = sb + 2 * (uint32_t)(lane / a.gchunks);
    const uint32_t lane16 = 16 * lane;
    uint32_t magic = 0x64006400u;
    asm volatile("" : "+v"(magic));
    int r = s0 / CPL, i = s0 % CPL;                         // row (within the workgroup) and chunk of the current slot
    auto read_slot = [&](int rr, int ii, int ri, u32x4& w, uint32_t& sc, u32x4 (&x)[4]) {
        w = lds_rd16(rg.addr(ri) + lane16);
        sc = lds_rdu16(sl + 2 * rr * ng + gstep * ii);
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) x[q4] = lds_rd16(xl + 4096 * ii + 16 * q4);
    };
    u32x4 cw, cx[4];
    uint32_t cs;
    if (rg.p <= rg.pmax) vm_wait<S - 1>(); else vm_wait_all();
    read_slot(r, i, rg.ri, cw, cs, cx);
    lgkm_wait_all();
    touch(cw);
    touch(cs);
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) touch(cx[q4]);
    float acc = 0.f;
    bool first_part = (i == 0);
    for (int k = 0; k < ns; ++k) {
        const bool more = k + 1 < ns;
        const int rn = Ring::next(rg.ri, S);
        const int i2 = (i + 1 == CPL) ? 0 : i + 1, r2 = (i + 1 == CPL) ? r + 1 : r;
        u32x4 nw, nx[4];
        uint32_t ns_ = 0u;
        if (more) {
            if (rg.p <= rg.pmax) vm_wait<S - 2>(); else vm_wait_all();
            read_slot(r2, i2, rn, nw, ns_, nx);
        }
        issue(rg.addr(rg.ri));                              // refill the slot just read into registers
        float slo = 0.f, shi = 0.f, lo0 = 0.f, lo1 = 0.f, hi0 = 0.f, hi1 = 0.f;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            const uint32_t x = cw[q4];
            const uint32_t y = x >> 8;
            const uint32_t p0 = bfi(0x000F000Fu, x, magic);
            const uint32_t p1 = bfi(0x00F000F0u, x, magic);
            const uint32_t p2 = bfi(0x000F000Fu, y, magic);
            const uint32_t p3 = bfi(0x00F000F0u, y, magic);
            const uint32_t x0 = cx[q4][0], x1 = cx[q4][1], x2 = cx[q4][2], x3 = cx[q4][3];
            float& lo = (q4 & 1) ? lo1 : lo0;
            float& hi = (q4 & 1) ? hi1 : hi0;
            lo = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p0), __builtin_bit_cast(half2_t, x0), lo, false);
            lo = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p2), __builtin_bit_cast(half2_t, x2), lo, false);
            hi = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p1), __builtin_bit_cast(half2_t, x1), hi, false);
            hi = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, p3), __builtin_bit_cast(half2_t, x3), hi, false);
            slo = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, x0), one2, slo, false);
            slo = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, x2), one2, slo, false);
            shi = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, x1), one2, shi, false);
            shi = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, x3), one2, shi, false);
        }
        const float dq = __builtin_fmaf(hi0 + hi1, 0.0625f, (lo0 + lo1) - (1032.0f * slo + 72.0f * shi));
        acc = __builtin_fmaf(f16_to_f32((uint16_t)cs), dq, acc);
        if (i + 1 == CPL || !more) {                        // this wave's part of row r is complete
            const float rs = wave_sum(acc);
            if (lane == 0) lds_wr4(res + 4 * (2 * r + (first_part ? 0 : 1)), rs);
            acc = 0.f;
            first_part = true;
        }
        if (more) {
            asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(acc)::"memory");
            touch(nw);
            touch(ns_);
            cw = nw;
            cs = ns_;
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                touch(nx[q4]);
                cx[q4] = nx[q4];
            }
        }
        ++rg.p;
        rg.ri = rn;
        r = r2;
        i = i2;
    }
}

// 2^x on the transcendental unit, without the library's range handling:
// softmax weights only take arguments <= 0, and weights below 2^-126 (flushed
// to zero) are far below the accuracy of the result.
__device__ __forceinline__ float exp2_raw(float x) { return __builtin_amdgcn_exp2f(x); }

// A chunk of tc (1..4) cache-row slot pairs: K and V of every pair are read
// into registers at once (one wait for the ring, one for LDS), then their
// refills are issued.  While the stream is not near its end, S - 2 tc younger
// ring positions stay in flight.
template <int S, class Issue>
__device__ __forceinline__ void att_read_chunk(Issue& issue, Ring& rg, int tc, u32x4 (&kw)[4], u32x4 (&vw)[4]) {
    static_assert(S >= 8, "a chunk of four pairs must fit the ring");
    const int lane16 = 16 * (threadIdx.x & 63);
    if (rg.p > rg.pmax) vm_wait_all();
    else if (tc == 4) vm_wait<S - 8>();
    else if (tc == 3) vm_wait<S - 6>();
    else if (tc == 2) vm_wait<S - 4>();
    else vm_wait<S - 2>();
    int ri = rg.ri;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        if (t < tc) {
            kw[t] = lds_rd16(rg.addr(ri) + lane16);
            ri = Ring::next(ri, S);
            vw[t] = lds_rd16(rg.addr(ri) + lane16);
            ri = Ring::next(ri, S);
        } else {
            kw[t] = u32x4{0u, 0u, 0u, 0u};
            vw[t] = u32x4{0u, 0u, 0u, 0u};
        }
    }
    lgkm_wait_all();
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        touch(kw[t]);
        touch(vw[t]);
    }
#pragma nounroll
    for (int t = 0; t < 2 * tc; ++t) {
        issue(rg.addr(rg.ri));
        rg.ri = Ring::next(rg.ri, S);
    }
    rg.p += 2 * tc;
}

// 8 cache values of one lane (16 bytes) as fp32.
template <bool BF16>
__device__ __forceinline__ void kv_to_f32(const u32x4& w, float (&f)[8]) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const uint32_t d = w[e];
        if constexpr (BF16) {
            f[2 * e] = __uint_as_float(d << 16);
            f[2 * e + 1] = __uint_as_float(d & 0xFFFF0000u);
        } else {
            f[2 * e] = f16_to_f32((uint16_t)(d & 0xFFFFu));
            f[2 * e + 1] = f16_to_f32((uint16_t)(d >> 16));
        }
    }
}

// This wave's cache rows of the layer's attention: T slot pairs (K then V),
// RPS rows per slot, LPR lanes per row.  Writes the wave's online-softmax
// partial (max, sum, unnormalized output per query head) to LDS part.
//
// The rows are taken in chunks of up to four slot pairs.  Within a chunk every
// score of every head is computed first (independent dot products and lane
// reductions), then one softmax update per head: the chunk's maximum, the
// weights of its rows and one rescale of the running sums, instead of one
// dependent update per row.  Each 16-lane row group keeps its own running
// (max, sum, output); the groups are combined at the end.
// rec (test support, null unless the layer's record is armed): the scores of
// the visible rows go to rec[h * keys + j], key j = j0 + t * RPS + lane / LPR of
// slot pair t, in natural-log units (q.k / sqrt(D)).
template <int GS, int D, int S, bool BF16, bool REC, class Issue>
__device__ __forceinline__ void att_seg_t(Issue& issue, Ring& rg, int T, uint32_t mbits, uint32_t qlds, uint32_t part,
                                          float* rec, int keys, int j0) {
    constexpr int LPR = AttGeo<D>::LPR;
    const int lane = threadIdx.x & 63;
    const int li = lane % LPR;
    float m[GS], l[GS], o[GS][8];
#pragma unroll
    for (int h = 0; h < GS; ++h) {
        m[h] = -INFINITY;
        l[h] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
    }
    if (T > 0) {
        u32x4 qv[GS][2];
#pragma unroll
        for (int h = 0; h < GS; ++h)
#pragma unroll
            for (int k = 0; k < 2; ++k) qv[h][k] = lds_rd16(qlds + 4 * (h * D + 8 * li + 4 * k));
        lgkm_wait_all();
        float qf[GS][8];
#pragma unroll
        for (int h = 0; h < GS; ++h)
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                touch(qv[h][k]);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t qe = qv[h][k][e];   // a scalar copy: bit_cast of a vector element reads element 0
                    qf[h][4 * k + e] = __builtin_bit_cast(float, qe);
                }
            }
        for (int t0 = 0; t0 < T; t0 += 4) {
            const int tc = min(4, T - t0);
            u32x4 kw[4], vw[4];
            att_read_chunk<S>(issue, rg, tc, kw, vw);
            // scores of every (row, head) of the chunk; rows not visible get -inf
            float sc[4][GS];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                float kf[8];
                kv_to_f32<BF16>(kw[t], kf);
                const bool vis = t < tc && ((mbits >> (t0 + t)) & 1u);
#pragma unroll
                for (int h = 0; h < GS; ++h) {
                    float sd = 0.f;
#pragma unroll
                    for (int e = 0; e < 8; ++e) sd = __builtin_fmaf(qf[h][e], kf[e], sd);
                    sd = group_sum<LPR>(sd);
                    sc[t][h] = vis ? sd : -INFINITY;
                    if constexpr (REC) {
                        const int j = j0 + (t0 + t) * AttGeo<D>::RPS + lane / LPR;
                        if (rec && vis && li == 0 && j < keys) rec[h * keys + j] = sd * 0.69314718055994531f;
                    }
                }
            }
            float vf[4][8];
#pragma unroll
            for (int t = 0; t < 4; ++t) kv_to_f32<BF16>(vw[t], vf[t]);
#pragma unroll
            for (int h = 0; h < GS; ++h) {
                float mn = m[h];
#pragma unroll
                for (int t = 0; t < 4; ++t) mn = fmaxf(mn, sc[t][h]);
                const float mref = (mn == -INFINITY) ? 0.f : mn;    // no visible row yet: nothing changes
                const float corr = exp2_raw(m[h] - mref);
                float p[4];
                float ls = 0.f;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    p[t] = exp2_raw(sc[t][h] - mref);
                    ls += p[t];
                }
                l[h] = __builtin_fmaf(l[h], corr, ls);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    float acc = o[h][e] * corr;
#pragma unroll
                    for (int t = 0; t < 4; ++t) acc = __builtin_fmaf(p[t], vf[t][e], acc);
                    o[h][e] = acc;
                }
                m[h] = mn;
            }
        }
        // merge the row groups (lanes LPR, 2 LPR, ... apart); for groups 16 and 32
        // lanes apart both partners of a pair receive the same two operands in the
        // same order, so they compute identical merges
#pragma unroll
        for (int h = 0; h < GS; ++h) {
#pragma unroll
            for (int sh = LPR; sh < 64; sh <<= 1) {
                float mA, mB, lA, lB;
                lane_pair(m[h], sh, mA, mB);
                lane_pair(l[h], sh, lA, lB);
                const float mn = fmaxf(mA, mB);
                const float mref = (mn == -INFINITY) ? 0.f : mn;
                const float wA = exp2_raw(mA - mref);
                const float wB = exp2_raw(mB - mref);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    float oA, oB;
                    lane_pair(o[h][e], sh, oA, oB);
                    o[h][e] = oA * wA + oB * wB;
                }
                l[h] = lA * wA + lB * wB;
                m[h] = mn;
            }
        }
    }
    const int cw = threadIdx.x >> 6;
    if (lane < LPR) {
#pragma unroll
        for (int h = 0; h < GS; ++h) {
            const uint32_t base = part + 4 * ((cw * GS + h) * (D + 4));
            lds_wr16(base + 16 + 32 * li, f32x4{o[h][0], o[h][1], o[h][2], o[h][3]});
            lds_wr16(base + 32 + 32 * li, f32x4{o[h][4], o[h][5], o[h][6], o[h][7]});
            if (li == 0) lds_wr16(base, f32x4{m[h], l[h], 0.f, 0.f});
        }
    }
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));

// 8 bytes per lane through the LDS transpose unit: in each 16-lane block, lane
// i receives element i % 4 of the reads of lanes i / 4, 4 + i / 4, 8 + i / 4
// and 12 + i / 4, in that order.
__device__ __forceinline__ u32x2 lds_rd8_tr(uint32_t a) {
    u32x2 v;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(a));
    return v;
}

// 16x16x32 and 16x16x16 products in the cache dtype, fp32 accumulation.
template <bool BF16>
__device__ __forceinline__ f32x4 mma_k32(const u32x4& A, const u32x4& B, f32x4 c) {
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, A), __builtin_bit_cast(bf16x8_t, B), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, A), __builtin_bit_cast(f16x8_t, B), c, 0, 0, 0);
}
template <bool BF16>
__device__ __forceinline__ f32x4 mma_k16(const u32x2& A, const u32x2& B, f32x4 c) {
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4_t, A), __builtin_bit_cast(i16x4_t, B), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4_t, A), __builtin_bit_cast(f16x4_t, B), c, 0, 0, 0);
}
template <bool BF16>
__device__ __forceinline__ float kv_value(uint16_t b) { return BF16 ? bf16_to_f32(b) : f16_to_f32(b); }
// Two floats rounded to the cache dtype (to nearest even), low half first.
template <bool BF16>
__device__ __forceinline__ uint32_t kv_pair(float lo, float hi) {
    if constexpr (BF16) {
        typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
        const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
        return __builtin_bit_cast(uint32_t, v);
    } else {
        return (uint32_t)f32_to_f16(lo) | ((uint32_t)f32_to_f16(hi) << 16);
    }
}

// The matrix-core form of the wave's attention (head_dim 128, at most four
// query heads per kv head): the rows go sixteen at a time (four slot pairs).
// The scores are computed transposed, S^T = K Q^T, with the 16 rows as the
// product's M rows and the heads as its N columns, each query entering as two
// cache-dtype terms (q = qh + qr, qr the rounding residual of qh), as in the
// per-layer attention.  Lane l then holds the scores of head l % 16 for rows
// 4 (l / 16) + j, j < 4, which is the A-operand layout of the 16x16x16 product
// P V: the weights are rounded to the cache dtype and used where they are.
// The V operand of 16-lane block b is slot pair b's V slot, transposed by the
// LDS read.  Running (max, sum) per head are kept per lane and combined over
// the four blocks at the end; the output accumulators hold head 4 (l / 16) + j
// in register j, so heads < 4 sit in lanes 0..15.
// qlds: the queries' two terms as written by the control wave (GS heads of qh,
// then GS heads of qr, each head ps_qb_stride(D) values).  mall: bit 4 t + r set when row r of slot
// pair t is visible.
template <int GS, int D, int S, bool BF16, bool REC, class Issue>
__device__ __forceinline__ void att_seg_m(Issue& issue, Ring& rg, int T, uint64_t mall, uint32_t qlds, uint32_t part,
                                          float* rec, int keys, int j0) {
    static_assert(D == 128 && GS >= 1 && GS <= 4 && S >= 8, "head_dim 128, up to four heads, two chunks of ring");
    constexpr int KB = D / 32;                 // 32-dim blocks of the score product
    constexpr int DB = D / 16;                 // 16-dim blocks of the output
    constexpr uint32_t RB = 2 * D;             // bytes per cache row
    const int lane = threadIdx.x & 63;
    const int i16 = lane & 15, b4 = lane >> 4;
    float m = -INFINITY, lsum = 0.f;
    f32x4 o[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d) o[d] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (T > 0) {
        // query operand: head i16 (zero for heads >= GS), dims 8 b4 + 32 kb .. + 7
        u32x4 qh[KB], qr[KB];
        {
            constexpr int QS = ps_qb_stride(D);
            const uint32_t qa = qlds + 2u * (uint32_t)((i16 < GS ? i16 : 0) * QS + 8 * b4);
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) {
                qh[kb] = lds_rd16(qa + 64u * kb);
                qr[kb] = lds_rd16(qa + (uint32_t)(GS * QS * 2) + 64u * kb);
            }
            lgkm_wait_all();
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) {
                touch(qh[kb]);
                touch(qr[kb]);
                if (i16 >= GS) {
                    qh[kb] = u32x4{0u, 0u, 0u, 0u};
                    qr[kb] = u32x4{0u, 0u, 0u, 0u};
                }
            }
        }
        for (int t0 = 0; t0 < T; t0 += 4) {
            const int tc = min(4, T - t0);
            if (rg.p > rg.pmax) vm_wait_all();
            else if (tc == 4) vm_wait<S - 8>();
            else if (tc == 3) vm_wait<S - 6>();
            else if (tc == 2) vm_wait<S - 4>();
            else vm_wait<S - 2>();
            // K operand: row i16 of the chunk (pair i16 / 4, row i16 % 4), dims 8 b4 + 32 kb;
            // V operand of block b4: pair b4's V slot.  Pairs past the chunk read the
            // chunk's last pair and are zeroed below (ring slots of other data may hold
            // any bits, and a zero weight times a NaN is a NaN).
            // (chunk c of key j sits at chunk c ^ (j mod 16) of its row)
            const int tk = i16 >> 2;
            int rk = rg.ri + 2 * min(tk, tc - 1);
            int rv = rg.ri + 2 * min(b4, tc - 1) + 1;
            rk -= rk >= S ? S : 0;
            rv -= rv >= S ? S : 0;
            const int swk = (j0 + 4 * (t0 + tk) + (i16 & 3)) & 15;   // key of this lane's K row
            const int swv = (j0 + 4 * (t0 + b4) + (i16 >> 2)) & 15;  // key of this lane's V read row
            const uint32_t ka = rg.addr(rk) + (uint32_t)(i16 & 3) * RB;
            const uint32_t va = rg.addr(rv) + (uint32_t)(i16 >> 2) * RB + 8u * (uint32_t)(i16 & 1);
            u32x4 kw[KB];
            u32x2 vf[DB];
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) kw[kb] = lds_rd16(ka + 16u * (uint32_t)((b4 + 4 * kb) ^ swk));
#pragma unroll
            for (int d = 0; d < DB; ++d) vf[d] = lds_rd8_tr(va + 16u * (uint32_t)((2 * d + ((i16 & 3) >> 1)) ^ swv));
            lgkm_wait_all();
            const bool kval = tk < tc, vval = b4 < tc;
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) {
                touch(kw[kb]);
                if (!kval) kw[kb] = u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int d = 0; d < DB; ++d) {
                touch(vf[d]);
                if (!vval) vf[d] = u32x2{0u, 0u};
            }
#pragma nounroll
            for (int t = 0; t < 2 * tc; ++t) {
                issue(rg.addr(rg.ri));
                rg.ri = Ring::next(rg.ri, S);
            }
            rg.p += 2 * tc;
            // scores of rows 4 b4 + j for head i16
            f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f}, sr = sc;       // two independent chains: qh and qr terms
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) {
                sc = mma_k32<BF16>(kw[kb], qh[kb], sc);
                sr = mma_k32<BF16>(kw[kb], qr[kb], sr);
            }
            sc += sr;
            const int sh = 4 * (t0 + b4);
            const uint32_t vis4 = sh < 64 ? (uint32_t)(mall >> sh) & 0xFu : 0u;
            float sv[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bool vis = i16 < GS && ((vis4 >> j) & 1u);
                sv[j] = vis ? sc[j] : -INFINITY;
                if constexpr (REC) {
                    const int key = j0 + sh + j;
                    if (rec && vis && key < keys) rec[i16 * keys + key] = sc[j] * 0.69314718055994531f;
                }
            }
            float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
            float xa, xb;
            lane_pair(mx, 16, xa, xb);
            mx = fmaxf(xa, xb);
            lane_pair(mx, 32, xa, xb);
            mx = fmaxf(xa, xb);
            const float mn = fmaxf(m, mx);
            const float mref = (mn == -INFINITY) ? 0.f : mn;    // no visible row yet: nothing changes
            const float corr = exp2_raw(m - mref);
            float p[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) p[j] = exp2_raw(sv[j] - mref);
            lsum = __builtin_fmaf(lsum, corr, (p[0] + p[1]) + (p[2] + p[3]));
            m = mn;
            const u32x2 pa = u32x2{kv_pair<BF16>(p[0], p[1]), kv_pair<BF16>(p[2], p[3])};
            if (t0 > 0 && __any(i16 < GS && corr != 1.f)) {     // some head's maximum moved (first chunk: o = 0)
                float cj[4];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    cj[j] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, corr), j));
#pragma unroll
                for (int d = 0; d < DB; ++d)
#pragma unroll
                    for (int j = 0; j < 4; ++j) o[d][j] *= cj[j];
            }
#pragma unroll
            for (int d = 0; d < DB; ++d) o[d] = mma_k16<BF16>(pa, vf[d], o[d]);
        }
        float la, lb2;
        lane_pair(lsum, 16, la, lb2);
        lsum = la + lb2;
        lane_pair(lsum, 32, la, lb2);
        lsum = la + lb2;
    }
    const int cw = threadIdx.x >> 6;
    if (b4 == 0) {
#pragma unroll
        for (int j = 0; j < GS; ++j) {
            const uint32_t base = part + 4 * ((cw * GS + j) * (D + 4));
#pragma unroll
            for (int d = 0; d < DB; ++d) lds_wr4(base + 16 + 4 * (16 * d + i16), o[d][j]);
        }
        if (i16 < GS) lds_wr16(part + 4 * ((cw * GS + i16) * (D + 4)), f32x4{m, lsum, 0.f, 0.f});
    }
}

template <int CPL_H, int CPL_Q, int CPL_F, int D, int GS, int S, bool KVB, bool REC>
__device__ __forceinline__ void compute_main(const PsArgs& a, uint32_t lb) {
    constexpr int LPR = AttGeo<D>::LPR, RPS = AttGeo<D>::RPS;
    const int lane = threadIdx.x & 63;
    const int cw = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int w = blockIdx.x;
    const int L = a.n_layers;

    const Rows rq_ = wave_rows(a.NQKV, a.rpw_qkv, w, cw);
    const Rows ro_ = wave_rows(a.H, a.rpw_h, w, cw);
    const Rows rg_ = wave_rows(2 * a.F, a.rpw_gu, w, cw);
    // attention rows of this wave: [j0, j0 + T * RPS) of this workgroup's split
    const ReqDev& rq = a.meta.reqs[0];
    const int P = rq.P;
    const bool has_att = w < a.Hkv * a.nsplit;
    const int T = has_att ? a.att_T : 0;
    const int g = has_att ? w / a.nsplit : 0;
    const int split = has_att ? w % a.nsplit : 0;
    const int sp0 = split * a.split_len, sp1 = min(P, sp0 + a.split_len);
    const int j0 = sp0 + cw * T * RPS;
    const int b = a.meta.items[0].slot;
    const u64 lstride_b = (u64)rq.S * a.Hkv * rq.cap * D * 2;
    const uint8_t* kbase = (const uint8_t*)rq.kc;
    const uint8_t* vbase = (const uint8_t*)rq.vc;
    uint32_t mbits = 0u;
    constexpr bool ATT_MMA = ps_att_mma(D, GS) && RPS * SK_TMAX <= 64;
    uint64_t mall = 0u;           // matrix-core form: every row r of slot pair t, at bit RPS t + r
    uint32_t aoff[SK_TMAX];       // per-lane byte offset of cache-row slot pair t within one layer
    {
        const uint8_t* mask = a.meta.masks + rq.mask_off + (size_t)b * rq.mask_len;
        const int16_t* tab = rq.table + (size_t)b * rq.cap;
#pragma unroll
        for (int t = 0; t < SK_TMAX; ++t) {
            const int j = j0 + t * RPS + lane / LPR;
            const bool valid = t < T && j < sp1;
            const int jj = valid ? j : 0;
            const int phys = valid ? (int)tab[jj] : b;
            if (valid && mask[jj] != 0) mbits |= 1u << t;
            // the matrix-core attention keeps row j's 16-byte chunk c at chunk c ^ (j mod 16)
            // of its LDS row (no two of a chunk's 16 rows on the same banks): this lane
            // loads the chunk that lands at its position
            const int ck = ATT_MMA ? ((lane % LPR) ^ (j & 15)) : lane % LPR;
            aoff[t] = (uint32_t)(((((u64)phys * a.Hkv + g) * rq.cap + jj) * D + 8 * ck) * 2);
            if constexpr (ATT_MMA) {
#pragma unroll
                for (int r = 0; r < RPS; ++r) {
                    const int jr = j0 + t * RPS + r;
                    if (t < T && jr < sp1 && mask[jr] != 0) mall |= 1ull << (RPS * t + r);
                }
            }
        }
    }
    // slots per segment of one layer: q|k|v rows, K/V slot pairs, o, gate|up, down rows
    // down rows: whole rows per wave when the input slice fits registers, else an even slot range
    // with one 1 KB block per compute wave (K = 2048 * SK_CW), wave cw takes block cw of every
    // down row of the workgroup: its input slice stays in registers for the whole segment
    constexpr bool XR_F = CPL_F <= 4;
    constexpr bool COL_F = CPL_F == SK_CW;
    const int wg_rows_h = max(0, min(a.H, (w + 1) * a.rpw_h) - w * a.rpw_h);
    const int kspw = kslot_per_wave(wg_rows_h, CPL_F);
    const int ks0 = min(wg_rows_h * CPL_F, cw * kspw);
    const int kns = min(wg_rows_h * CPL_F, ks0 + kspw) - ks0;
    const int n0 = rq_.count * CPL_H, n1 = 2 * T, n2 = ro_.count * CPL_Q, n3 = rg_.count * CPL_H;
    const int n4 = COL_F ? wg_rows_h : XR_F ? ro_.count * CPL_F : kns;
    const int total = (n0 + n1 + n2 + n3 + n4) * L;
    // The weight rows of one wave in one segment are contiguous in the row layout
    // (kc = 64 * CPL chunks per row), so a segment streams one block of 1 KB slots.
    // Stream state: segment gs of layer gl, gleft slots left in it.  In a weight
    // segment every slot but the last is issued by the fast path (gfast counts
    // them); the last one, the attention slots and the end of the stream take
    // the general path, which also moves to the next segment.
    int gl = 0, gs = -1, gleft = 0, gt = 0, gfast = 0;
    const uint8_t* gptr = nullptr;
    u64 gstride = SK_SLOT;                                  // bytes between a segment's consecutive slots
    auto next_seg = [&]() {
        do {
            if (++gs == 5) {
                gs = 0;
                ++gl;
            }
        } while (gl < L && (gs == 0 ? n0 : gs == 1 ? n1 : gs == 2 ? n2 : gs == 3 ? n3 : n4) == 0);
        if (gl >= L) {
            gleft = 0;
            gfast = 0;
            return;
        }
        gleft = gs == 0 ? n0 : gs == 1 ? n1 : gs == 2 ? n2 : gs == 3 ? n3 : n4;
        gt = 0;
        gstride = (COL_F && gs == 4) ? (u64)a.kc_f * 16 : (u64)SK_SLOT;
        if (gs == 0) gptr = a.wb[0] + gl * a.wl[0] + (u64)rq_.first * a.kc_h * 16;
        else if (gs == 2) gptr = a.wb[1] + gl * a.wl[1] + (u64)ro_.first * a.kc_q * 16;
        else if (gs == 3) gptr = a.wb[2] + gl * a.wl[2] + (u64)rg_.first * a.kc_h * 16;
        else if (gs == 4)
            gptr = a.wb[3] + gl * a.wl[3] +
                   (COL_F  ? (u64)w * a.rpw_h * a.kc_f * 16 + (u64)cw * SK_SLOT
                    : XR_F ? (u64)ro_.first * a.kc_f * 16
                           : (u64)w * a.rpw_h * a.kc_f * 16 + (u64)ks0 * SK_SLOT);
        if (gs != 1) {
            gfast = gleft - 1;
            gleft = 1;
        }
    };
    const uint32_t lane16 = 16u * (uint32_t)lane;
    auto issue_general = [&](uint32_t dst) {
        if (gleft == 0) return;                             // past the end of the stream: nothing to load
        if (gs == 1) {
            const int t = gt >> 1;
            uint32_t off = aoff[0];
#pragma unroll
            for (int k = 1; k < SK_TMAX; ++k) {
                int kk = k;
                asm volatile("" : "+s"(kk));          // keeps this a select chain, not an indexed array
                off = (t == kk) ? aoff[k] : off;
            }
            dma16(((gt & 1) ? vbase : kbase) + (u64)gl * lstride_b + off, dst);
            ++gt;
        } else {
            dma16(gptr + lane16, dst);
        }
        if (--gleft == 0) next_seg();
    };
    auto issue = [&](uint32_t dst) {
        if (gfast > 0) {
            --gfast;
            dma16(gptr + lane16, dst);
            gptr += gstride;
        } else {
            issue_general(dst);
        }
    };
    const uint32_t ring = lb + (uint32_t)(cw * S * SK_SLOT);
    next_seg();
    vm_wait_all();                                          // table and mask reads are done
    for (int k = 0; k < S; ++k) issue(ring + (uint32_t)k * SK_SLOT);

    Ring rg{ring, 0, 0, total - S};
    for (int l = 0; l < L; ++l) {
        wg_barrier();                                       // input of q|k|v is staged
        gemv_seg<CPL_H, S>(a, issue, rg, rq_.count, rq_.local, a.ng_h, lb + a.l_sb0, lb + a.l_xs, lb + a.l_res);
        wg_barrier();                                       // q|k|v rows are in LDS
        wg_barrier();                                       // q and the new row are staged
        cstamp(a, lb + a.l_dbg, 0);
        float* rec = nullptr;
        if constexpr (REC)
            if (l == a.dbg_layer && has_att) rec = a.dbg_logits + (size_t)g * GS * a.dbg_keys;
        if constexpr (ATT_MMA)
            att_seg_m<GS, D, S, KVB, REC>(issue, rg, T, mall, lb + a.l_qb, lb + a.l_part, rec, a.dbg_keys, j0);
        else
            att_seg_t<GS, D, S, KVB, REC>(issue, rg, T, mbits, lb + a.l_q, lb + a.l_part, rec, a.dbg_keys, j0);
        cstamp(a, lb + a.l_dbg, 1);
        wg_barrier();                                       // wave partials are in LDS
        wg_barrier();                                       // this workgroup's merge is done: polling starts now
        {                                                   // the attention output of every head
            constexpr int NTO = (CPL_Q * 512 + 64 * SK_CW - 1) / (64 * SK_CW);   // Hq*D <= 2048 CPL_Q
            stage_pairs<NTO>(a, a.ll_o, a.QD / 4, cw, a.ll_epoch + PS_LL_PER_LAYER * l + 3, lb + a.l_xs, true);
        }
        wg_barrier();                                       // attention output is staged
        gemv_seg<CPL_Q, S>(a, issue, rg, ro_.count, ro_.local, a.ng_q, lb + a.l_sb1, lb + a.l_xs, lb + a.l_res);
        wg_barrier();                                       // o rows are in LDS: the input is free
        stage_x_words<CPL_H>(a, cw, a.ll_epoch + PS_LL_PER_LAYER * l + 4, lb + a.l_xs, true);
        wg_barrier();                                       // RMSNorm(x) is staged
        cstamp(a, lb + a.l_dbg, 2);
        gemv_seg<CPL_H, S>(a, issue, rg, rg_.count, rg_.local, a.ng_h, lb + a.l_sb0, lb + a.l_xs, lb + a.l_res);
        cstamp(a, lb + a.l_dbg, 3);
        wg_barrier();                                       // gate|up rows are in LDS: the input is free
        // this wave's share of the SwiGLU output (ring loads already in flight complete first)
        {
            constexpr int NTA = (CPL_F * 512 + 64 * SK_CW - 1) / (64 * SK_CW);   // F <= 2048 CPL_F
            stage_pairs<NTA>(a, a.ll_act, a.F / 4, cw, a.ll_epoch + PS_LL_PER_LAYER * l + 5, lb + a.l_xs, true);
        }
        wg_barrier();                                       // SwiGLU output is staged
        cstamp(a, lb + a.l_dbg, 4);
        if constexpr (COL_F)
            gemv_seg<1, S>(a, issue, rg, wg_rows_h, 0, a.ng_f, lb + a.l_sb1 + (uint32_t)(cw * (128 / a.gchunks)),
                           lb + a.l_xs + 4096u * cw, lb + a.l_res + 4u * cw * a.rpw_h);
        else if constexpr (XR_F)
            gemv_seg<CPL_F, S>(a, issue, rg, ro_.count, ro_.local, a.ng_f, lb + a.l_sb1, lb + a.l_xs, lb + a.l_res);
        else
            gemv_seg_k<CPL_F, S>(a, issue, rg, ks0, kns, a.ng_f, lb + a.l_sb1, lb + a.l_xs, lb + a.l_res);
        cstamp(a, lb + a.l_dbg, 5);
        wg_barrier();                                       // down rows are in LDS: the input is free
        if (l + 1 < L) stage_x_words<CPL_H>(a, cw, a.ll_epoch + PS_LL_PER_LAYER * l + 6, lb + a.l_xs, true);
    }
}

// ------------------------------------------------------------------ control wave

// Scale rows [first, first + count) of a matrix with ng groups per row into LDS
// (direct loads of 1 KB; the allocation is padded so the last one stays in bounds).
__device__ __forceinline__ void load_scales(const uint16_t* s, int first, int count, int ng, uint32_t dst) {
    const int lane = threadIdx.x & 63;
    const uint8_t* src = (const uint8_t*)(s + (size_t)first * ng);
    const int bytes = count * ng * 2;
    for (int off = 0; off < bytes; off += SK_SLOT) dma16(src + off + 16 * lane, dst + off);
}

// Input of the first q|k|v GEMV: the stage input h (K values of dtype src_dt,
// written before the launch) -> h * rsqrt(mean(h^2) + eps) * gamma as fp16 in
// LDS xs, padding up to kpad zeroed; returns the RMSNorm scale.
template <int NT>
__device__ __forceinline__ float stage_norm(const void* src, int src_dt, int K, int kpad, const uint8_t* gl,
                                            int gamma_dt, float eps, uint8_t* xs) {
    const int lane = threadIdx.x & 63;
    const int n4 = K / 4;
    f32x4 v[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int it = lane + 64 * t;
        const u32x2 h = *(const u32x2*)((const uint16_t*)src + 4 * (it < n4 ? it : 0));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t wd = h[e >> 1];
            v[t][e] = half_bits_to_f32((uint16_t)((e & 1) ? (wd >> 16) : (wd & 0xFFFFu)), src_dt);
        }
    }
    float ss = 0.f;
#pragma unroll
    for (int t = 0; t < NT; ++t)
        if (lane + 64 * t < n4) ss += v[t][0] * v[t][0] + v[t][1] * v[t][1] + v[t][2] * v[t][2] + v[t][3] * v[t][3];
    const float rs = rsqrtf(wave_sum(ss) / (float)K + eps);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int it = lane + 64 * t;
        if (it < n4) {
            const u32x2 gv = *(const u32x2*)(gl + 8 * it);
            float y[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t wd = gv[e >> 1];
                y[e] = (v[t][e] * rs) * half_bits_to_f32((uint16_t)((e & 1) ? (wd >> 16) : (wd & 0xFFFFu)), gamma_dt);
            }
            *(u32x2*)(xs + 8 * it) = u32x2{pack_f16x2(y[0], y[1]), pack_f16x2(y[2], y[3])};
        }
    }
    for (int it = n4 + lane; it < kpad / 4; it += 64) *(u32x2*)(xs + 8 * it) = u32x2{0u, 0u};
    return rs;
}

__device__ __forceinline__ void zero_pad(int K, int kpad, uint8_t* xs) {
    const int lane = threadIdx.x & 63;
    for (int it = K / 8 + lane; it < kpad / 8; it += 64) *(f32x4*)(xs + 16 * it) = f32x4{0.f, 0.f, 0.f, 0.f};
}

__device__ __forceinline__ void lds_wr8(uint32_t a, u32x2 v) {
    asm volatile("ds_write_b64 %0, %1" ::"v"(a), "v"(v) : "memory");
}

// ---- the residual stream between workgroups
//
// RMSNorm(x) W^T = rs * ((x * gamma) W^T) with the scalar rs = rsqrt(mean(x^2) + eps):
// each row owner publishes u = fp16(x * gamma * c) for its rows together with
// the rows' sum of squares, and a consumer applies rs / c to the GEMV results.
// c is the previous normalization's rs, identical in every workgroup, which
// keeps u in the range the normalized input would have.  The exchange buffer
// holds H 4-byte words (u) followed by one 8-byte word per workgroup (its sum
// of squares; the count is rounded up to even).

__device__ __forceinline__ int ss_words(int nwg) { return (nwg + 1) & ~1; }

__device__ __forceinline__ void publish_x(const PsArgs& a, int xr0, int nxr, float xrow, float gamma, float c,
                                          uint32_t flag) {
    const int lane = threadIdx.x & 63;
    if (lane < nxr) ll_store16(a.ll_x + xr0 + lane, f32_to_f16(xrow * gamma * c), flag);
    const float ss = wave_sum(lane < nxr ? xrow * xrow : 0.f);
    u64* sw = (u64*)(a.ll_x + a.H);
    if (lane == 0) ll_store(sw + blockIdx.x, __float_as_uint(ss), flag);
    if (lane == 1 && (gridDim.x & 1) && blockIdx.x == gridDim.x - 1) ll_store(sw + gridDim.x, 0u, flag);
}

// The published u, polled by the compute waves (compute wave wv of SK_CW takes
// pieces lane + 64 (wv + SK_CW t)) into LDS xs: a wave that only polls is not
// held up by the acknowledgement of stores of its own.
template <int CPL_H>
__device__ __forceinline__ bool stage_x_words(const PsArgs& a, int wv, uint32_t flag, uint32_t xs, bool ok) {
    constexpr int NTX = (CPL_H * 512 + 64 * SK_CW - 1) / (64 * SK_CW);   // pieces (four u) per lane: H <= 2048 CPL_H
    const int lane = fresh_lane();
    const __amdgpu_buffer_rsrc_t r = make_rsrc(a.ll_x, (size_t)a.H * 4);
    int off[NTX];
    uint32_t use = 0u;
#pragma unroll
    for (int t = 0; t < NTX; ++t) {
        const int it = lane + 64 * (wv + SK_CW * t);
        const bool u = it < a.H / 4;
        off[t] = u ? 16 * it : 0;
        use |= (u ? 1u : 0u) << t;
    }
    return ll_wait<NTX, NTX>(a, r, off, use, flag, [&](int i, const u32x4& pc) {
        const uint32_t w0 = pc[0], w1 = pc[1], w2 = pc[2], w3 = pc[3];
        lds_wr8(xs + 8 * (lane + 64 * (wv + SK_CW * i)), u32x2{(w0 & 0xFFFFu) | (w1 << 16), (w2 & 0xFFFFu) | (w3 << 16)});
    }, ok);
}

// rs from the workgroups' published sums of squares (added in a fixed order);
// the control wave, which published, polls only these.
__device__ __forceinline__ float stage_x_rs(const PsArgs& a, uint32_t flag, bool& ok, int tl, int tw) {
    constexpr int NSP = 2;                 // pieces (two sums) per lane: up to 256 workgroups
    const int lane = fresh_lane();
    const int nss = ss_words(gridDim.x);
    const __amdgpu_buffer_rsrc_t r = make_rsrc(a.ll_x, (size_t)a.H * 4 + (size_t)nss * 8);
    int off[NSP];
    uint32_t use = 0u;
#pragma unroll
    for (int t = 0; t < NSP; ++t) {
        const int it = lane + 64 * t;
        const bool u = it < nss / 2;
        off[t] = u ? 4 * a.H + 16 * it : 0;
        use |= (u ? 1u : 0u) << t;
    }
    float ssv[2 * NSP];
#pragma unroll
    for (int j = 0; j < 2 * NSP; ++j) ssv[j] = 0.f;
    ok = ll_wait<NSP>(a, r, off, use, flag, [&](int i, const u32x4& pc) {
        const uint32_t w0 = pc[0], w2 = pc[2];
        ssv[2 * i] = __uint_as_float(w0);
        ssv[2 * i + 1] = __uint_as_float(w2);
    }, ok, tl, tw);
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < 2 * NSP; ++j) ss += ssv[j];
    return rsqrtf(wave_sum(ss) / (float)a.H + a.eps);
}

// A buffer of fp16 pairs in 8-byte flag words (attention output, SwiGLU output),
// polled by NW compute waves into LDS xs: wave wv of them takes pieces (four
// values) lane + 64 (wv + NW t), t < NT.
template <int NT, int NW = SK_CW>
__device__ __forceinline__ bool stage_pairs(const PsArgs& a, const u64* buf, int npieces, int wv, uint32_t flag,
                                            uint32_t xs, bool ok) {
    const int lane = fresh_lane();
    const __amdgpu_buffer_rsrc_t r = make_rsrc(buf, (size_t)npieces * 16);
    int off[NT];
    uint32_t use = 0u;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int it = lane + 64 * (wv + NW * t);
        const bool u = it < npieces;
        off[t] = u ? 16 * it : 0;
        use |= (u ? 1u : 0u) << t;
    }
    return ll_wait<NT>(a, r, off, use, flag, [&](int i, const u32x4& pc) {
        const uint32_t p0 = pc[0], p1 = pc[2];
        lds_wr8(xs + 8 * (lane + 64 * (wv + NW * i)), u32x2{p0, p1});
    }, ok);
}

// v combined (op: commutative, exact for max) over the lanes congruent to this
// one modulo ch (a power of two, 1..64): lane exchanges within 4 lanes, DPP
// rotations within a 16-lane row, then the swaps of 16- and 32-lane halves.
// N values at once: one uniform branch per step.
template <int N, class Op>
__device__ __forceinline__ void split_combine(float (&v)[N], int ch, Op op) {
    if (ch <= 1)
#pragma unroll
        for (int i = 0; i < N; ++i) v[i] = op(v[i], dpp_f<0xB1>(v[i]));   // quad_perm [1,0,3,2]: lane ^ 1
    if (ch <= 2)
#pragma unroll
        for (int i = 0; i < N; ++i) v[i] = op(v[i], dpp_f<0x4E>(v[i]));   // quad_perm [2,3,0,1]: lane ^ 2
    if (ch <= 4)
#pragma unroll
        for (int i = 0; i < N; ++i) v[i] = op(v[i], dpp_f<0x124>(v[i]));  // row_ror:4
    if (ch <= 8)
#pragma unroll
        for (int i = 0; i < N; ++i) v[i] = op(v[i], dpp_f<0x128>(v[i]));  // row_ror:8: the class within the row
    if (ch <= 16)
#pragma unroll
        for (int i = 0; i < N; ++i) {
            float a, b;
            lane_pair(v[i], 16, a, b);
            v[i] = op(a, b);
        }
    if (ch <= 32)
#pragma unroll
        for (int i = 0; i < N; ++i) {
            float a, b;
            lane_pair(v[i], 32, a, b);
            v[i] = op(a, b);
        }
}

// Split merge (control wave of each attention workgroup): every split of a
// kv head reads the partials (max, sum, outputs) of all the head group's splits
// for its own 1/nsplit slice of the group's outputs, combines them in a fixed
// butterfly order and publishes that slice of the attention output.
template <int GS, int D>
__device__ __forceinline__ void merge_slices(const PsArgs& a, int g, int split, uint32_t f_part, uint32_t f_o, int l) {
    const int SL = GS * D / a.nsplit;                 // outputs per slice (multiple of 8)
    const int CH = SL / 8;                            // 8-output chunks per slice
    const int ml = fresh_lane();
    const int s2 = ml / CH, c = ml % CH;              // lane: one split's chunk of the slice
    const bool act = s2 < a.nsplit;
    const int o0 = split * SL + 8 * c;                // first output of the chunk within the head group
    const int hh = o0 / D, dd = o0 % D;
    constexpr int PREC = ps_part_words(D);
    const __amdgpu_buffer_rsrc_t r = make_rsrc(a.ll_part, (size_t)a.Hkv * a.nsplit * GS * PREC * 8);
    const int base = act ? (int)((((size_t)g * a.nsplit + s2) * GS + hh) * PREC) * 8 : 0;
    const int off[3] = {base, base + 8 * (2 + dd / 2), base + 8 * (2 + dd / 2) + 16};
    u32x4 pv[3];
    ll_wait<3>(a, r, off, act ? 0x7u : 0u, f_part, [&](int i, const u32x4& pc) { pv[i] = pc; }, true, l, 1);
    float ms = -INFINITY, ls = 0.f, ov[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) ov[e] = 0.f;
    if (act) {
        const uint32_t m0 = pv[0][0], l0 = pv[0][2];
        ms = __uint_as_float(m0);
        ls = __uint_as_float(l0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t x = pv[1 + j / 2][2 * (j % 2)];      // fp16 pair of outputs 2j, 2j + 1
            ov[2 * j] = f16_to_f32((uint16_t)(x & 0xFFFFu));
            ov[2 * j + 1] = f16_to_f32((uint16_t)(x >> 16));
        }
    }
    // combine the splits: lanes c, c + CH, c + 2 CH, ... (CH a power of two), by
    // lane exchanges that stay in registers; every lane of a class gets the same
    // maximum, and lanes 0..CH-1 sums taken in a fixed order.  A split's weight is
    // 2^(m - M) times its sum (its outputs are normalized by that sum).
    float mv[1] = {ms};
    split_combine(mv, CH, [](float x, float y) { return fmaxf(x, y); });
    const float wgt = (ms == -INFINITY) ? 0.f : exp2f(ms - mv[0]) * ls;
    float sv[9];
    sv[8] = wgt;
#pragma unroll
    for (int e = 0; e < 8; ++e) sv[e] = ov[e] * wgt;
    split_combine(sv, CH, [](float x, float y) { return x + y; });
    const float Ls = sv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) ov[e] = sv[e];
    if (act && s2 == 0) {
        const float inv = 1.0f / Ls;
        const __amdgpu_buffer_rsrc_t orr = make_rsrc(a.ll_o, (size_t)a.QD * 4);
        const int ob = ((g * GS + hh) * D + dd) * 4;      // byte offset of output dd's word (dd: a multiple of 8)
#pragma unroll
        for (int e = 0; e < 8; e += 4)
            ll_store2(orr, ob + 4 * e, pack_f16x2(ov[e] * inv, ov[e + 1] * inv),
                      pack_f16x2(ov[e + 2] * inv, ov[e + 3] * inv), f_o);
    }
}

// The layer table, read through the constant address space: it is not written
// during the launch, so its (uniform) reads are scalar loads, which do not wait
// behind this wave's outstanding global stores and direct-to-LDS loads.
typedef const __attribute__((address_space(4))) PsLayer CPsLayer;

template <int CPL_H, int CPL_Q, int CPL_F, int D, int GS, int S, bool KVB, bool REC>
__device__ __forceinline__ void control_main(const PsArgs& a, uint8_t* smem) {
    const int lane = threadIdx.x & 63;
    CPsLayer* lays = (CPsLayer*)a.layers;
    const int w = blockIdx.x;
    const uint32_t lb = lds_addr(smem);
    uint8_t* xs = smem + a.l_xs;
    const float* res = (const float*)(smem + a.l_res);
    float* qs = (float*)(smem + a.l_q);
    uint32_t* qhb = (uint32_t*)(smem + a.l_qb);   // query pairs as two cache-dtype terms: qh, then qr
    float* nkv = (float*)(smem + a.l_nkv);
    const float* part = (const float*)(smem + a.l_part);
    const float2* rope = (const float2*)(smem + a.l_rope);
    constexpr int NT_H = CPL_H * 8;          // float4 items per lane of a K = H input (K padded to 2048 * CPL_H)
    constexpr int OPL = GS * D / 64;         // merged outputs per lane
    constexpr int LPH = D / OPL;             // lanes per query head in the merge
    static_assert(OPL == 2 || OPL == 4 || OPL == 8, "merge layout");

    const ReqDev& rq = a.meta.reqs[0];
    const int P = rq.P;
    const int b = a.meta.items[0].slot;
    const int pos = a.meta.positions[0];
    const uint8_t* mask = a.meta.masks + rq.mask_off + (size_t)b * rq.mask_len;
    const bool has_att = w < a.Hkv * a.nsplit;
    const int g = has_att ? w / a.nsplit : 0;
    const int split = has_att ? w % a.nsplit : 0;
    const bool owns_new = has_att && split == a.nsplit - 1;
    const bool new_vis = owns_new && mask[P] != 0;           // this forward's row is visible to its own query
    const int KVD = a.Hkv * D;
    const size_t lstride = (size_t)rq.S * a.Hkv * rq.cap * D;
    const int hq = lane / LPH, d0 = (lane % LPH) * OPL;     // merge lane layout

    // own rows of the residual stream (o and down rows of this workgroup), one per lane
    const int xr0 = w * a.rpw_h;
    const int nxr = max(0, min(a.H, xr0 + a.rpw_h) - xr0);
    float xrow = 0.f;
    if (lane < nxr) xrow = half_bits_to_f32(((const uint16_t*)a.hidden_in)[xr0 + lane], a.act_dt);
    if (lane < D / 2) ((float2*)rope)[lane] = a.rope[(size_t)pos * (D / 2) + lane];
    load_scales(lays[0].qkv.s, w * a.rpw_qkv, max(0, min(a.NQKV, (w + 1) * a.rpw_qkv) - w * a.rpw_qkv), a.ng_h,
                lb + a.l_sb0);
    vm_wait_all();
    // c: scale of the last published residual (the last RMSNorm scale); mq, mg: the
    // factors rs / c applied to the q|k|v and gate|up results.  The first
    // normalization reads the stage input and its RMSNorm weights from memory.
    float c = stage_norm<NT_H>(a.hidden_in, a.act_dt, a.H, a.kc_h * 32, (const uint8_t*)lays[0].attn_norm, a.act_dt,
                               a.eps, xs);
    float mq = 1.f, mg = 1.f;
    bool ok = true;
    vm_wait_all();
    wg_barrier();                                             // q|k|v input staged

    for (int l = 0; l < a.n_layers; ++l) {
        const CPsLayer& Ly = lays[l];
        const bool last = (l == a.n_layers - 1);
        // flag numbers of this layer's exchanges
        const uint32_t f_qkv = a.ll_epoch + PS_LL_PER_LAYER * l + 1, f_part = f_qkv + 1, f_o = f_qkv + 2,
                       f_xo = f_qkv + 3, f_act = f_qkv + 4, f_xd = f_qkv + 5;
        stamp(a, l, 0);
        load_scales(Ly.o.s, xr0, nxr, a.ng_q, lb + a.l_sb1);
        // RMSNorm weights of the own rows, for the residuals published after o and after down
        float gam_f = 0.f, gam_a = 0.f;
        if (lane < nxr) {
            gam_f = half_bits_to_f32(Ly.ffn_norm[xr0 + lane], a.act_dt);
            if (!last) gam_a = half_bits_to_f32(lays[l + 1].attn_norm[xr0 + lane], a.act_dt);
        }
        if (l > 0) {
            // rs of the residual published after the previous layer's down product,
            // polled while the compute waves run this layer's q|k|v rows.  No
            // workgroup can rewrite these words before this one publishes q|k|v.
            const float rs = stage_x_rs(a, a.ll_epoch + PS_LL_PER_LAYER * (l - 1) + 6, ok, l - 1, 5);
            mq = rs / c;
            c = rs;
        }
        wg_barrier();                                         // q|k|v rows are in LDS
        stamp(a, l, 1);
        // ---- RMSNorm scale and rotary embedding of q and k (rows 2d, 2d + 1 of a head are d, d + D/2), as flag words
        {
            const int r0 = w * a.rpw_qkv;
            const int n = max(0, min(a.NQKV, r0 + a.rpw_qkv) - r0);
            for (int k = lane; k < n / 2; k += 64) {
                const int pr = r0 + 2 * k;
                const int hb = pr / D, d = (pr % D) / 2;
                float lo = res[2 * k] * mq, hi = res[2 * k + 1] * mq;
                if (hb < a.Hq + a.Hkv) {
                    const float2 cs = rope[d];
                    const float l2 = lo * cs.x - hi * cs.y;
                    hi = hi * cs.x + lo * cs.y;
                    lo = l2;
                }
                ll_store(&a.ll_qkv[hb * D + d], __float_as_uint(lo), f_qkv);
                ll_store(&a.ll_qkv[hb * D + d + D / 2], __float_as_uint(hi), f_qkv);
            }
        }
        stamp(a, l, 2);
        // ---- stage this split's query heads and, for the last split, this forward's cache row
        if (has_att) {
            constexpr int NQP = GS * D / 128 > 0 ? GS * D / 128 : 1;   // 16-byte pieces (two values) of q per lane
            constexpr int NKP = D / 128 > 0 ? D / 128 : 1;             // pieces of the new k (and of v) per lane
            constexpr int NP = NQP + 2 * NKP;
            const int lane = fresh_lane();
            const __amdgpu_buffer_rsrc_t r = make_rsrc(a.ll_qkv, (size_t)a.NQKV * 8);
            int off[NP];
            uint32_t use = 0u;
#pragma unroll
            for (int t = 0; t < NQP; ++t) {
                const int it = lane + 64 * t;
                const bool u = it < GS * D / 2;
                off[t] = u ? (g * GS * D + 2 * it) * 8 : 0;
                use |= (u ? 1u : 0u) << t;
            }
#pragma unroll
            for (int t = 0; t < NKP; ++t) {
                const int it = lane + 64 * t;
                const bool u = owns_new && it < D / 2;
                off[NQP + t] = u ? (a.QD + g * D + 2 * it) * 8 : 0;
                off[NQP + NKP + t] = u ? (a.QD + KVD + g * D + 2 * it) * 8 : 0;
                use |= (u ? 1u : 0u) << (NQP + t);
                use |= (u ? 1u : 0u) << (NQP + NKP + t);
            }
            u32x4 kv[2 * NKP];                                 // new k, v pieces
            ok = ll_wait<NP>(a, r, off, use, f_qkv, [&](int i, const u32x4& pc) {
                const uint32_t p0 = pc[0], p1 = pc[2];
                if (i < NQP) {
                    const float y0 = __uint_as_float(p0) * a.qscale, y1 = __uint_as_float(p1) * a.qscale;
                    *(float2*)(qs + 2 * (lane + 64 * i)) = float2{y0, y1};
                    if constexpr (ps_att_mma(D, GS)) {              // the matrix-core attention's query terms
                        const uint32_t hi = kv_pair<KVB>(y0, y1);
                        const float r0 = y0 - kv_value<KVB>((uint16_t)(hi & 0xFFFFu));
                        const float r1 = y1 - kv_value<KVB>((uint16_t)(hi >> 16));
                        constexpr int QS = ps_qb_stride(D);          // values per head in LDS
                        const int vi = 2 * (lane + 64 * i);          // first value of the pair
                        const int wo = (vi / D) * (QS / 2) + (vi % D) / 2;
                        qhb[wo] = hi;
                        qhb[GS * QS / 2 + wo] = kv_pair<KVB>(r0, r1);
                    }
                } else {
                    kv[i - NQP] = pc;
                }
            }, ok, l, 0);
            if (owns_new) {
                uint16_t* kl = rq.kc + (size_t)l * lstride + (((size_t)b * a.Hkv + g) * rq.cap + P) * D;
                uint16_t* vl = rq.vc + (size_t)l * lstride + (((size_t)b * a.Hkv + g) * rq.cap + P) * D;
#pragma unroll
                for (int t = 0; t < NKP; ++t) {
                    const int it = lane + 64 * t;
                    if (it < D / 2) {
                        const uint32_t k0 = kv[t][0], k1 = kv[t][2];
                        const uint32_t v0 = kv[NKP + t][0], v1 = kv[NKP + t][2];
                        const uint16_t kb0 = to_half_bits(__uint_as_float(k0), a.kv_dt), kb1 = to_half_bits(__uint_as_float(k1), a.kv_dt);
                        const uint16_t vb0 = to_half_bits(__uint_as_float(v0), a.kv_dt), vb1 = to_half_bits(__uint_as_float(v1), a.kv_dt);
                        *(uint32_t*)(kl + 2 * it) = (uint32_t)kb0 | ((uint32_t)kb1 << 16);
                        *(uint32_t*)(vl + 2 * it) = (uint32_t)vb0 | ((uint32_t)vb1 << 16);
                        *(float2*)(nkv + 2 * it) = float2{half_bits_to_f32(kb0, a.kv_dt), half_bits_to_f32(kb1, a.kv_dt)};
                        *(float2*)(nkv + D + 2 * it) = float2{half_bits_to_f32(vb0, a.kv_dt), half_bits_to_f32(vb1, a.kv_dt)};
                    }
                }
                if (l == 0 && g == 0 && lane == 0) rq.table[(size_t)b * rq.cap + P] = (int16_t)b;
            }
        }
        wg_barrier();                                         // q and the new row are staged
        wg_barrier();                                         // wave partials are in LDS
        stamp(a, l, 3);
        // ---- merge the waves (and the new row) into this split's partial; the last split merges the splits
        if (has_att) {
            // every wave's (max, sum) of head hq and this lane's OPL outputs of it, and
            // the new row's query and cache values, read with one wait
            constexpr int NR = OPL >= 4 ? OPL / 4 : 1;         // 16-byte reads per OPL values (OPL = 2: one 8-byte read)
            u32x4 pml[SK_CW], po[SK_CW][NR], qn[NR], kn[NR], vn[NR];
            u32x2 po2[SK_CW], qn2 = u32x2{0u, 0u}, kn2 = qn2, vn2 = qn2;
#pragma unroll
            for (int r = 0; r < NR; ++r) qn[r] = kn[r] = vn[r] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int c = 0; c < SK_CW; ++c) {
                const uint32_t pa = lb + a.l_part + 4u * (uint32_t)((c * GS + hq) * (D + 4));
                pml[c] = lds_rd16(pa);
                if constexpr (OPL >= 4) {
#pragma unroll
                    for (int r = 0; r < NR; ++r) po[c][r] = lds_rd16(pa + 16u + 4u * d0 + 16u * r);
                } else {
                    po2[c] = lds_rd8(pa + 16u + 4u * d0);
                }
            }
            if (new_vis) {
                const uint32_t qa = lb + a.l_q + 4u * (uint32_t)(hq * D + d0), na = lb + a.l_nkv + 4u * d0;
                if constexpr (OPL >= 4) {
#pragma unroll
                    for (int r = 0; r < NR; ++r) {
                        qn[r] = lds_rd16(qa + 16u * r);
                        kn[r] = lds_rd16(na + 16u * r);
                        vn[r] = lds_rd16(na + 4u * D + 16u * r);
                    }
                } else {
                    qn2 = lds_rd8(qa);
                    kn2 = lds_rd8(na);
                    vn2 = lds_rd8(na + 4u * D);
                }
            }
            lgkm_wait_all();
            float pm[SK_CW], pl[SK_CW], pov[SK_CW][OPL], qv[OPL], kv_[OPL], vv[OPL];
#pragma unroll
            for (int c = 0; c < SK_CW; ++c) {
                touch(pml[c]);
                const uint32_t m0 = pml[c][0], l0 = pml[c][1];
                pm[c] = __uint_as_float(m0);
                pl[c] = __uint_as_float(l0);
                if constexpr (OPL >= 4) {
#pragma unroll
                    for (int r = 0; r < NR; ++r) {
                        touch(po[c][r]);
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const uint32_t x = po[c][r][e];
                            pov[c][4 * r + e] = __uint_as_float(x);
                        }
                    }
                } else {
                    touch(po2[c]);
                    const uint32_t x0 = po2[c][0], x1 = po2[c][1];
                    pov[c][0] = __uint_as_float(x0);
                    pov[c][1] = __uint_as_float(x1);
                }
            }
            if constexpr (OPL >= 4) {
#pragma unroll
                for (int r = 0; r < NR; ++r) {
                    touch(qn[r]);
                    touch(kn[r]);
                    touch(vn[r]);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t xq = qn[r][e], xk = kn[r][e], xv = vn[r][e];
                        qv[4 * r + e] = __uint_as_float(xq);
                        kv_[4 * r + e] = __uint_as_float(xk);
                        vv[4 * r + e] = __uint_as_float(xv);
                    }
                }
            } else {
                touch(qn2);
                touch(kn2);
                touch(vn2);
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const uint32_t xq = qn2[e], xk = kn2[e], xv = vn2[e];
                    qv[e] = __uint_as_float(xq);
                    kv_[e] = __uint_as_float(xk);
                    vv[e] = __uint_as_float(xv);
                }
            }
            float s_new = -INFINITY;
            if (new_vis) {
                float sd = 0.f;
#pragma unroll
                for (int e = 0; e < OPL; ++e) sd += qv[e] * kv_[e];
                sd = (LPH == 16) ? group_sum<16>(sd) : (LPH == 8) ? group_sum<8>(sd) : sd;
                if constexpr (LPH == 32) {
                    sd = group_sum<16>(sd);
                    sd += dpp_rows<0x142, 0xA>(sd);                       // row 1 += row 0, row 3 += row 2
                    sd = __shfl(sd, (lane & 32) + 31);
                }
                s_new = sd;
                if constexpr (REC)
                    if (l == a.dbg_layer && (lane % LPH) == 0 && P < a.dbg_keys)
                        a.dbg_logits[(size_t)(g * GS + hq) * a.dbg_keys + P] = sd * 0.69314718055994531f;
            }
            if constexpr (REC)
                if (l == a.dbg_layer && split == 0)                   // this kv head's rotated queries
                    for (int idx = lane; idx < GS * D; idx += 64) a.dbg_q[(size_t)g * GS * D + idx] = qs[idx] / a.qscale;
            float mx = s_new;
#pragma unroll
            for (int c = 0; c < SK_CW; ++c) mx = fmaxf(mx, pm[c]);
            float L = 0.f, O[OPL];
#pragma unroll
            for (int e = 0; e < OPL; ++e) O[e] = 0.f;
            if (s_new != -INFINITY) {
                const float wn = exp2f(s_new - mx);
                L = wn;
#pragma unroll
                for (int e = 0; e < OPL; ++e) O[e] = wn * vv[e];
            }
#pragma unroll
            for (int c = 0; c < SK_CW; ++c) {
                const float wc = (pm[c] == -INFINITY) ? 0.f : exp2f(pm[c] - mx);
                L += wc * pl[c];
#pragma unroll
                for (int e = 0; e < OPL; ++e) O[e] += wc * pov[c][e];
            }
            {   // (max, sum), and the outputs divided by the sum and rounded to fp16 (the
                // precision the merged output is published in), as pairs of flag words
                constexpr int PREC = ps_part_words(D);
                const __amdgpu_buffer_rsrc_t pr = make_rsrc(a.ll_part, (size_t)a.Hkv * a.nsplit * GS * PREC * 8);
                const int pb = (((g * a.nsplit + split) * GS + hq) * PREC) * 8;
                const float inv = L > 0.f ? 1.0f / L : 0.f;
                if constexpr (OPL >= 4) {
#pragma unroll
                    for (int e = 0; e < OPL; e += 4)
                        ll_store2(pr, pb + 8 * (2 + (d0 + e) / 2), pack_f16x2(O[e] * inv, O[e + 1] * inv),
                                  pack_f16x2(O[e + 2] * inv, O[e + 3] * inv), f_part);
                } else {
                    ll_store(a.ll_part + pb / 8 + 2 + d0 / 2, pack_f16x2(O[0] * inv, O[1] * inv), f_part);
                }
                if (d0 == 0) ll_store2(pr, pb, __float_as_uint(mx), __float_as_uint(L), f_part);
            }
            const u64 t_pub = a.trace ? wall_clock64() : 0ull;
            merge_slices<GS, D>(a, g, split, f_part, f_o, l);
            if (a.trace && lane == 0) a.trace[((size_t)w * a.n_layers + l) * PS_TRACE_PER_LAYER + 31] = t_pub;
        }
        stamp(a, l, 4);
        wg_barrier();                                         // merge done: the compute waves poll the attention output
        // gate|up scales (q|k|v finished with this buffer), loaded after the exchange
        // waits of the attention, which they would hold up, and awaited while the
        // compute waves stage the attention output
        load_scales(Ly.gu.s, w * a.rpw_gu, max(0, min(2 * a.F, (w + 1) * a.rpw_gu) - w * a.rpw_gu), a.ng_h, lb + a.l_sb0);
        zero_pad(a.QD, a.kc_q * 32, xs);                      // (they stage it)
        vm_wait_all();
        wg_barrier();                                         // attention output staged
        wg_barrier();                                         // o rows are in LDS
        stamp(a, l, 5);
        // ---- x += o Wo^T (own rows), published for the ffn RMSNorm
        if (lane < nxr) xrow += res[lane];
        publish_x(a, xr0, nxr, xrow, gam_f, c, f_xo);
        stamp(a, l, 6);
        zero_pad(a.H, a.kc_h * 32, xs);                       // the compute waves stage the published x
        wg_barrier();                                         // RMSNorm(x) staged
        load_scales(Ly.d.s, xr0, nxr, a.ng_f, lb + a.l_sb1);   // o finished with this buffer
        {
            // rs of the published x, needed by the SwiGLU epilogue only: polled while
            // the compute waves run gate|up.  No workgroup can rewrite these words
            // before this one publishes its SwiGLU output, which comes later.
            const float rs = stage_x_rs(a, f_xo, ok, l, 3);
            mg = rs / c;
            c = rs;
        }
        wg_barrier();                                         // gate|up rows are in LDS
        stamp(a, l, 7);
        // ---- act = silu(gate) * up, two outputs per flag word
        {
            const int r0 = w * a.rpw_gu;
            const int n = max(0, min(2 * a.F, r0 + a.rpw_gu) - r0);
            for (int k = lane; k < n / 4; k += 64) {
                float y[2];
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const float gt = res[4 * k + 2 * e] * mg, up = res[4 * k + 2 * e + 1] * mg;
                    y[e] = (gt / (1.0f + expf(-gt))) * up;
                }
                ll_store(a.ll_act + r0 / 4 + k, pack_f16x2(y[0], y[1]), f_act);
            }
        }
        stamp(a, l, 8);
        zero_pad(a.F, a.kc_f * 32, xs);                       // the compute waves stage the SwiGLU output
        wg_barrier();                                         // SwiGLU output staged
        if (!last) {
            const CPsLayer& Ln = lays[l + 1];
            load_scales(Ln.qkv.s, w * a.rpw_qkv, max(0, min(a.NQKV, (w + 1) * a.rpw_qkv) - w * a.rpw_qkv), a.ng_h,
                        lb + a.l_sb0);
        }
        wg_barrier();                                         // down rows are in LDS
        stamp(a, l, 9);
        if (a.trace && lane < 6)
            a.trace[((size_t)blockIdx.x * a.n_layers + l) * PS_TRACE_PER_LAYER + 10 + lane] = ((const u64*)(smem + a.l_dbg))[lane];
        // ---- x += act Wd^T (own rows); the last layer writes hidden_out
        if (lane < nxr) {
            if constexpr (CPL_F == SK_CW) {                   // one partial per compute wave, added in wave order
                float d = 0.f;
#pragma unroll
                for (int c = 0; c < SK_CW; ++c) d += res[c * a.rpw_h + lane];
                xrow += d;
            } else if constexpr (CPL_F <= 4) {
                xrow += res[lane];
            } else {                                          // rows shared by two waves have two partials
                const int kspw = kslot_per_wave(nxr, CPL_F);
                const bool two = (lane * CPL_F) / kspw != (lane * CPL_F + CPL_F - 1) / kspw;
                xrow += two ? res[2 * lane] + res[2 * lane + 1] : res[2 * lane];
            }
            if (last) ((uint16_t*)a.hidden_out)[xr0 + lane] = to_half_bits(xrow, a.act_dt);
        }
        if (!last) {
            publish_x(a, xr0, nxr, xrow, gam_a, c, f_xd);
            zero_pad(a.H, a.kc_h * 32, xs);
            wg_barrier();                                     // next layer's q|k|v input staged
            // its rs is polled at the start of the next layer (needed by the q|k|v epilogue)
        }
    }
}

// REC: the variant that also writes the armed attention record (a.dbg_q,
// a.dbg_logits); the plain variant carries none of that code.
template <int CPL_H, int CPL_Q, int CPL_F, int D, int GS, int S, bool KVB, bool REC>
__global__ __launch_bounds__(SK_THREADS) void stage_stream_kernel(PsArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    if ((threadIdx.x >> 6) < SK_CW)
        compute_main<CPL_H, CPL_Q, CPL_F, D, GS, S, KVB, REC>(a, lds_addr(smem));
    else
        control_main<CPL_H, CPL_Q, CPL_F, D, GS, S, KVB, REC>(a, smem);
}

// ------------------------------------------------------------------ host side

// Instantiations: (K / 2048 for K = H, Hq*D, F), head_dim, query heads per kv
// head, ring slots, KV cache in bf16 (1) or fp16 (0).
#define PS_SHAPES(X)                     \
    X(2, 2, 7, 128, 4, 16, 1)   /* Llama-3.1-8B layers, bf16 cache */ \
    X(1, 1, 1, 64, 2, 14, 0)    /* small test stages, fp16 cache */

#define PS_KEY(H_, Q_, F_, D_, G_, K_) (cpl_h == H_ && cpl_q == Q_ && cpl_f == F_ && D == D_ && gs == G_ && kvb == K_)
#define PS_KERNEL(H_, Q_, F_, D_, G_, S_, K_) stage_stream_kernel<H_, Q_, F_, D_, G_, S_, (K_ != 0), false>
#define PS_KERNEL_REC(H_, Q_, F_, D_, G_, S_, K_) stage_stream_kernel<H_, Q_, F_, D_, G_, S_, (K_ != 0), true>

bool ps_supported(int cpl_h, int cpl_q, int cpl_f, int D, int gs, int kvb) {
#define PS_MATCH(H_, Q_, F_, D_, G_, S_, K_) \
    if (PS_KEY(H_, Q_, F_, D_, G_, K_)) return true;
    PS_SHAPES(PS_MATCH)
#undef PS_MATCH
    return false;
}

int ps_slots(int cpl_h, int cpl_q, int cpl_f, int D, int gs, int kvb) {
#define PS_MATCH(H_, Q_, F_, D_, G_, S_, K_) \
    if (PS_KEY(H_, Q_, F_, D_, G_, K_)) return S_;
    PS_SHAPES(PS_MATCH)
#undef PS_MATCH
    return 0;
}

static size_t ps_private_of(const void* fn) {
    hipFuncAttributes at{};
    if (hipFuncGetAttributes(&at, fn) != hipSuccess) {
        (void)hipGetLastError();
        return (size_t)-1;
    }
    return at.localSizeBytes;
}

size_t ps_private_bytes(int cpl_h, int cpl_q, int cpl_f, int D, int gs, int kvb) {
#define PS_MATCH(H_, Q_, F_, D_, G_, S_, K_) \
    if (PS_KEY(H_, Q_, F_, D_, G_, K_)) return ps_private_of((const void*)PS_KERNEL(H_, Q_, F_, D_, G_, S_, K_));
    PS_SHAPES(PS_MATCH)
#undef PS_MATCH
    return (size_t)-1;
}

static int ps_blocks_of(const void* fn, size_t lds) {
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, SK_THREADS, lds) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    return n;
}

int ps_blocks_per_cu(int cpl_h, int cpl_q, int cpl_f, int D, int gs, int kvb, size_t lds) {
#define PS_MATCH(H_, Q_, F_, D_, G_, S_, K_) \
    if (PS_KEY(H_, Q_, F_, D_, G_, K_)) return ps_blocks_of((const void*)PS_KERNEL(H_, Q_, F_, D_, G_, S_, K_), lds);
    PS_SHAPES(PS_MATCH)
#undef PS_MATCH
    return 0;
}

static hipError_t launch_ps(const void* fn, const PsArgs& a, int nwg, size_t lds, bool coop, hipStream_t st) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    PsArgs copy = a;
    void* args[] = {&copy};
    if (coop) return hipLaunchCooperativeKernel(fn, dim3(nwg), dim3(SK_THREADS), args, (unsigned)lds, st);
    return hipLaunchKernel(fn, dim3(nwg), dim3(SK_THREADS), args, (unsigned)lds, st);
}

hipError_t launch_persistent(const PsArgs& a, int cpl_h, int cpl_q, int cpl_f, int D, int gs, int kvb, int nwg, size_t lds,
                             bool coop, hipStream_t st) {
#define PS_MATCH(H_, Q_, F_, D_, G_, S_, K_)                                                                      \
    if (PS_KEY(H_, Q_, F_, D_, G_, K_))                                                                          \
        return launch_ps(a.dbg_logits ? (const void*)PS_KERNEL_REC(H_, Q_, F_, D_, G_, S_, K_)                   \
                                      : (const void*)PS_KERNEL(H_, Q_, F_, D_, G_, S_, K_), a, nwg, lds, coop, st);
    PS_SHAPES(PS_MATCH)
#undef PS_MATCH
    return hipErrorInvalidValue;
}
#undef PS_KEY
#undef PS_KERNEL
#undef PS_KERNEL_REC

// Destination row of source row r: row_off + r (map 0), 2r (map 1, gate),
// 2r + 1 (map 2, up), or row_off + the rotary-pair order inside each head of
// head_dim rows (map 3: d -> 2d for d < D/2, d -> 2(d - D/2) + 1 otherwise).
__host__ __device__ __forceinline__ int row_dest(int r, int row_off, int row_map, int head_dim) {
    if (row_map == 1) return 2 * r;
    if (row_map == 2) return 2 * r + 1;
    if (row_map == 3) {
        const int h = r / head_dim, d = r % head_dim, half = head_dim / 2;
        return row_off + h * head_dim + (d < half ? 2 * d : 2 * (d - half) + 1);
    }
    return row_off + r;
}

__global__ void repack_rows_kernel(const uint8_t* __restrict__ q, const uint16_t* __restrict__ s, int n, int k, int g,
                                   uint8_t* __restrict__ w_out, uint16_t* __restrict__ s_out, int kc, int ng,
                                   int row_off, int row_map, int head_dim) {
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= (size_t)n * kc) return;
    const int r = (int)(idx / kc), c = (int)(idx % kc);
    const int kb = (k + 1) / 2;
    const int dr = row_dest(r, row_off, row_map, head_dim);
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
                              int kc, int ng, int row_off, int row_map, int head_dim, hipStream_t st) {
    const size_t nc = (size_t)n * kc;
    repack_rows_kernel<<<dim3((unsigned)((nc + 255) / 256)), dim3(256), 0, st>>>(q, s, n, k, g, w_out, s_out, kc, ng,
                                                                                row_off, row_map, head_dim);
    return hipGetLastError();
}

__global__ void dequant_rows_kernel(PsMat m, int kc, int ng, int gchunks, int k, int row_off, int row_map, int n_rows,
                                    int head_dim, float* __restrict__ out) {
    const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
    if (idx >= (size_t)n_rows * kc) return;
    const int r = (int)(idx / kc), c = (int)(idx % kc);
    const int dr = row_dest(r, row_off, row_map, head_dim);
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
                               int head_dim, float* out, hipStream_t st) {
    const size_t nc = (size_t)n_rows * kc;
    dequant_rows_kernel<<<dim3((unsigned)((nc + 255) / 256)), dim3(256), 0, st>>>(m, kc, ng, gchunks, k, row_off, row_map,
                                                                                  n_rows, head_dim, out);
    return hipGetLastError();
}

}  // namespace stg
