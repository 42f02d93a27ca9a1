// Internal declarations shared by the host runtime and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace stg {

constexpr int TILE_ROWS = 64;        // weight rows per tile: one row per lane of a wave
constexpr int CHUNK_K = 32;          // k values per 16-byte chunk (32 nibbles)
constexpr int MAX_ROWS = 64;         // activation rows per forward
constexpr int GEMV_MAX_M = 8;        // rows one GEMV launch handles
constexpr int GEMV_MAX_CPS = 64;     // chunks per workgroup: 4 waves x at most 16 chunks
constexpr int ATTN_MAX_SPLITS = 64;  // KV splits per (slot, kv head)
constexpr int ATTN_MIN_SPLIT = 32;   // fewest keys per split
constexpr int KGROUPS = 16;          // 16-lane key groups per attention workgroup

enum Dt : int { DT_F32 = 0, DT_F16 = 1, DT_BF16 = 2 };

// INT4 matrix in the tiled device layout.
//   w: [ntiles][nchunk][64 lanes] x 16 bytes; lane r of tile t holds row 64t+r,
//      chunk c holds k in [32c, 32c+32).  Nibble order inside each dword
//      (k = 8d .. 8d+7 of the chunk, d = dword index): bits 0-3 -> k, 16-19 -> k+1,
//      4-7 -> k+2, 20-23 -> k+3, 8-11 -> k+4, 24-27 -> k+5, 12-15 -> k+6,
//      28-31 -> k+7, so that mask-and-or with 0x6400 yields fp16 pairs of
//      consecutive k.  Codes are offset binary (u = q + 8); padding rows and
//      columns hold u = 8 (q = 0).
//   s: [ntiles][ngroups][64] fp16 scales (0 for padding rows).
struct PackedMat {
    const uint8_t* w;
    const uint16_t* s;
    int n, k, ntiles, nchunk, ngroups, gchunks;  // gchunks = group_size / 32
};

// Per-request metadata on the device (one forward).
struct ReqDev {
    int P, n, S, row0, cap, mask_off, mask_len, item0;
    uint16_t* kc;        // K cache, layer 0 base: [L][S][Hkv][cap][D]
    uint16_t* vc;        // V cache
    int16_t* table;      // current beam table [S][cap] (physical slot of each row)
};

struct ItemDev {         // one (request, slot) pair: the unit of the attention grid
    int req, slot;
};

struct MetaDev {
    const ReqDev* reqs;
    const ItemDev* items;
    const int* positions;   // [M]: rotary position of each activation row
    const uint8_t* masks;   // concatenated [S][P+n] per request
    int n_items, M;
};

enum GemvRms : int { RMS_NONE = 0, RMS_FULLROW = 1, RMS_PARTIALS = 2 };
enum GemvEpi : int { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2 };

struct GemvArgs {
    PackedMat W;
    const void* in; int in_dt; int in_ld;          // input rows [M][K]
    const uint16_t* gamma; int gamma_dt;           // RMSNorm weight [K]
    int rms; float eps;
    const float* ssq_in; int ssq_tiles;            // [ssq_tiles][M] sums of squares
    int M;
    int ksplit, cps;
    float* partial; unsigned* counters;            // [ksplit][M][ntiles*64], [ntiles]
    int epi;
    float* out; int out_ld;                        // STORE: out, RESID: new x, SWIGLU: act
    const void* resid; int resid_dt; int resid_ld; // RESID source
    float* ssq_out;                                // RESID: [ntiles][M]
    void* out_act; int out_act_dt; int out_act_ld; // RESID: optional copy in act dtype
    int n_valid;                                   // SWIGLU: F
};

struct AttnArgs {
    const float* qkv; int qkv_ld;
    float* out; int out_ld;
    MetaDev meta;
    const float2* rope;      // [max_positions][D/2] (cos, sin)
    int layer, Hq, Hkv, kv_dt;
    float qscale;            // log2(e) / sqrt(D)
    float* part; unsigned* counters;
    int nsplit_max;
};

// Kernel launchers (kernels.hip).
hipError_t launch_repack(const uint8_t* q, const uint16_t* s, int n, int k, int g,
                         uint8_t* w_out, uint16_t* s_out, int ntiles, int nchunk, int ngroups,
                         int row_off, int row_map, hipStream_t st);
hipError_t launch_gemv(const GemvArgs& a, hipStream_t st);
hipError_t launch_attention(const AttnArgs& a, int head_dim, int rows_per_item_max, hipStream_t st);
hipError_t launch_table_gather(const int16_t* src, int16_t* dst, const int* beam, int S, int cap, int P, hipStream_t st);
hipError_t launch_kv_append(uint16_t* kc, uint16_t* vc, int16_t* table, const uint16_t* k, const uint16_t* v,
                            int L, int S, int Hkv, int cap, int D, int P, int n, hipStream_t st);
hipError_t launch_kv_read(const uint16_t* kc, const uint16_t* vc, const int16_t* table, int layer, int slot,
                          int start, int count, int S, int Hkv, int cap, int D, uint16_t* k_out, uint16_t* v_out,
                          hipStream_t st);
hipError_t launch_dequant(const PackedMat& m, int row_off, int row_map, int n_rows, float* out, hipStream_t st);

}  // namespace stg
