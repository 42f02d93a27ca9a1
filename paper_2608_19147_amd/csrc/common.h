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
constexpr int ATTN_MIN_SPLIT = 256;  // fewest keys per split
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
    int rowmask_off;     // per-query-row masks [S][n][mask_len] in MetaDev::masks, or -1 (slot masks only)
    int splits;          // most attention splits per (slot, kv head): a function of the request alone
    uint16_t* kc;        // K cache, layer 0 base: [L][S][Hkv][cap][D]
    uint16_t* vc;        // V cache
    int16_t* table;      // current beam table [S][cap] (physical slot of each row)
};

struct ItemDev {         // one (request, slot) pair: the unit of the attention grid
    int req, slot;
    ReqDev rq;           // a copy of the request's record (one load instead of two dependent ones)
};

struct MetaDev {
    const ReqDev* reqs;
    const ItemDev* items;
    const int* positions;   // [M]: rotary position of each activation row
    const int* row_item;    // [M]: item (request slot) of each activation row
    const uint8_t* masks;   // concatenated [S][P+n] per request, then the requests' per-row masks
    int n_items, M, n_req;
};

enum GemvRms : int { RMS_NONE = 0, RMS_FULLROW = 1, RMS_PARTIALS = 2 };
enum GemvEpi : int { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_TOP1 = 3 };

struct GemvArgs {
    PackedMat W;
    const void* in; int in_dt; int in_ld;          // input rows [M][K]
    const uint16_t* gamma; int gamma_dt;           // RMSNorm weight [K]
    int rms; float eps;
    const float* ssq_in; int ssq_tiles;            // [M][ssq_tiles] sums of squares
    int M;
    int ksplit, cps;
    float* partial; unsigned* counters;            // [ksplit][M][ntiles*64], [ntiles]
    int epi;
    float* out; int out_ld;                        // STORE: out, RESID: new x, SWIGLU: act
    const void* resid; int resid_dt; int resid_ld; // RESID source
    float* ssq_out;                                // RESID: [M][ntiles]
    void* out_act; int out_act_dt; int out_act_ld; // RESID: optional copy in act dtype
    int n_valid;                                   // SWIGLU: F
    // prepared-operand products (gemm_bp_kernel): input rows in matrix-core form
    const uint16_t* bp_in; const float* bc_in;     // [M][kp] codes, [M][kp/32] corrections
    const float* cb_in;                            // norm 1: scale c each row was prepared with
    int norm;                                      // 0: none, 1: deferred RMSNorm (factor rs / c), 2: prepared normalized
    int kp, kg;                                    // prepared row stride; groups of 128 k per wave
    float* rs_out;                                 // norm 1: rs of each row, for the next residual product
    uint16_t* bp_out; float* bc_out; float* cb_out;  // RESID / SWIGLU: the next product's input
    const uint16_t* gamma_next; int gamma_next_dt; // RESID: RMSNorm weight of the next product
    const float* rs_in;                            // RESID: scale c to prepare with (previous rs)
    float4* top1_part;                             // TOP1: [M][ntiles] (max, index bits, sum of exp(v - max), 0)
};

// Prefill product (gemm_pf_kernel): W [N][K] (tiled) times the prepared rows of
// n tokens, kept as 64-row blocks of the prepared-operand layout (block b at
// bp + b * bp_blk halves, its corrections at bc + b * bc_blk floats).
struct PfArgs {
    PackedMat W;
    const uint16_t* bp; const float* bc; size_t bp_blk, bc_blk;
    int n;                                         // tokens
    int epi;                                       // EPI_STORE, EPI_RESID, EPI_SWIGLU
    float* out; int out_ld;                        // STORE: out; RESID: new x; SWIGLU: act (fp32)
    const void* resid; int resid_dt; int resid_ld; // RESID source (may be out itself)
    void* out_act; int out_act_dt; int out_act_ld; // RESID: optional copy in the act dtype
    int n_valid;                                   // SWIGLU: F
    int nwt, ntb;                                  // groups of 4 weight tiles, 64-token blocks
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
    int vector_path;         // 1: attn_kernel (vector units) instead of attn_mma_kernel
    uint16_t* bp_out; float* bc_out; int kp;   // the attention output also in prepared form (o product input, 64-row blocks)
    int no_append;           // the rows of this forward are already in the cache (prefill): do not write them
    int dma;                 // 1: cache rows by direct loads (attn_dma_kernel) where the launch allows it: every
                             // split at most 1024 keys, per-row masks of at most 8 KB per split, at most 256
                             // query vectors per kv head
    // test support (null unless armed): the rotated queries [M][Hq][D] and the
    // scores q.k / sqrt(D) of every visible key [M][Hq][dbg_keys]
    float* dbg_q; float* dbg_logits; int dbg_keys;
};

// ---- single-launch stage forward (persistent.hip)
constexpr int PS_MAX_M = 1;          // rows of one single-launch forward (decode of one slot)
constexpr int PS_KCHUNK = 2048;      // row-layout K is padded to a multiple of this
constexpr int SK_CW = 7;             // compute waves per workgroup; with the control wave, two waves per SIMD
constexpr int SK_SLOT = 1024;        // bytes per ring slot: one 16-byte load per lane
constexpr int SK_TMAX = 16;          // cache-row slot pairs (K, V) per compute wave per layer

// Row layout: w [N][kc][16 bytes] (chunk c of row n holds k in [32c, 32c+32),
// same nibble order as PackedMat), s [N][ng] fp16 scales.  The q|k|v matrix
// stores each head's rows d and d + D/2 next to each other (row 2d and 2d + 1
// of the head's block), so one workgroup owns both rows of every rotary pair.
struct PsMat {
    const uint8_t* w;
    const uint16_t* s;
};

struct PsLayer {
    PsMat qkv, o, gu, d;                 // gu rows interleave gate (2f) and up (2f+1)
    const uint16_t* attn_norm;
    const uint16_t* ffn_norm;
};

struct PsArgs {
    const PsLayer* layers;               // device array
    // Code rows of each matrix kind (q|k|v, o, gate|up, down) for all layers in
    // one allocation: layer l's rows start at wb[m] + l * wl[m] (equal to
    // layers[l].<m>.w), so the compute waves form stream addresses without loads.
    const uint8_t* wb[4];
    unsigned long long wl[4];
    int n_layers;
    int H, Hq, Hkv, F, QD, NQKV;
    int kc_h, kc_q, kc_f;                // chunks per row for K = H, Hq*D, F
    int ng_h, ng_q, ng_f;                // scale groups per row
    int gchunks;                         // chunks per scale group
    float eps;
    int act_dt, kv_dt;
    const void* hidden_in;
    void* hidden_out;
    int rpw_qkv, rpw_h, rpw_gu;          // rows per workgroup: q|k|v, o and down, gate|up
    unsigned* ll_x;                      // [H] 4-byte flag words (fp16): published residual rows, then
                                         // [nwg rounded up to even] 8-byte flag words (fp32): their sums of squares
    unsigned long long* ll_qkv;          // [NQKV] flag words (fp32 values): rotated q, rotated k, v
    unsigned long long* ll_o;            // [QD / 2] flag words (fp16 pairs): attention output
    unsigned long long* ll_act;          // [F / 2] flag words (fp16 pairs): SwiGLU output
    MetaDev meta;
    const float2* rope;
    float qscale;                        // log2(e) / sqrt(D)
    int nsplit, split_len, att_T;        // splits per kv head (power of two), cache rows per split, slot pairs per wave
    unsigned long long* ll_part;         // [Hkv][nsplit][Hq/Hkv][ps_part_words(D)] flag words: max, sum (fp32),
                                         // then the outputs / sum as fp16 pairs
    unsigned ll_epoch;                   // flag numbers used by earlier launches (PS_LL_PER_LAYER per layer)
    unsigned* err;                       // set when an exchange wait gives up
    unsigned spin_limit;                 // polling passes after which an exchange wait gives up
    unsigned long long* trace;           // optional [nwg][n_layers][PS_TRACE_PER_LAYER] real-time stamps
    // test support (null unless armed): layer dbg_layer's rotated query [Hq][D]
    // and the score q.k / sqrt(D) of every key the row sees, [Hq][dbg_keys]
    float* dbg_q; float* dbg_logits; int dbg_keys, dbg_layer;
    // LDS byte offsets
    int l_xs, l_sb0, l_sb1, l_res, l_q, l_qb, l_nkv, l_part, l_rope, l_dbg, l_end;
};
constexpr int PS_LL_PER_LAYER = 6;      // flag-word exchanges per layer: q|k|v, split partials, attention
                                        // output, residual after o, SwiGLU output, residual after down
constexpr int PS_TRACE_PER_LAYER = 40;   // 10 control-wave boundaries, 6 from compute wave 0, 6 exchange pass
                                         // counts, 6 exchange end times, 3 first-pass times, partial published,
                                         // 6 first-pass issue times, 2 spare

// Values per head in the stream kernel's LDS copy of the query terms: D plus
// 32 of padding, so the four heads a 16-byte read meets start 64 bytes apart
// in the LDS banks.
constexpr int ps_qb_stride(int D) { return D + 32; }

// Flag words of one split's partial of one query head: max, sum, D / 2 pairs.
constexpr int ps_part_words(int D) { return 2 + D / 2; }

// The stream kernel's attention runs on the matrix cores for head_dim 128 and
// at most four query heads per kv head.
constexpr bool ps_att_mma(int D, int gs) { return D == 128 && gs <= 4; }

// LDS layout of the stream kernel with `slots` ring slots per compute wave;
// returns the total bytes.
inline int ps_layout(PsArgs& a, int slots, int D, int gs) {
    auto up = [](int v, int m) { return (v + m - 1) / m * m; };
    const int kcmax = a.kc_h > a.kc_q ? (a.kc_h > a.kc_f ? a.kc_h : a.kc_f) : (a.kc_q > a.kc_f ? a.kc_q : a.kc_f);
    int sb = a.rpw_qkv * a.ng_h;
    sb = sb > a.rpw_h * a.ng_q ? sb : a.rpw_h * a.ng_q;
    sb = sb > a.rpw_gu * a.ng_h ? sb : a.rpw_gu * a.ng_h;
    sb = sb > a.rpw_h * a.ng_f ? sb : a.rpw_h * a.ng_f;
    sb = up(sb * 2, SK_SLOT);
    int rows = a.rpw_qkv > 2 * a.rpw_h ? a.rpw_qkv : 2 * a.rpw_h;   // down rows may carry two partials
    rows = rows > a.rpw_gu ? rows : a.rpw_gu;
    rows = rows > SK_CW * a.rpw_h ? rows : SK_CW * a.rpw_h;         // or one per compute wave
    int off = SK_CW * slots * SK_SLOT;
    a.l_xs = off;   off += kcmax * 64;                                // staged GEMV input (fp16)
    a.l_sb0 = off;  off += sb;
    a.l_sb1 = off;  off += sb;
    a.l_res = off;  off += up(rows * 4, 16);
    a.l_q = off;    off += gs * D * 4;
    a.l_nkv = off;  off += 2 * D * 4;
    // the compute waves' attention partials and the queries as two cache-dtype
    // terms live only between the q|k|v product (the last reader of the staged
    // input) and the staging of the o input, so they share the staged-input
    // region when they fit
    const int part_b = up(SK_CW * gs * (D + 4) * 4, 16);
    const int qb_b = ps_att_mma(D, gs) ? 2 * gs * ps_qb_stride(D) * 2 : 0;
    if (part_b + qb_b <= kcmax * 64) {
        a.l_part = a.l_xs;
        a.l_qb = a.l_xs + part_b;
    } else {
        a.l_part = off; off += part_b;
        a.l_qb = off;   off += up(qb_b, 16);
    }
    a.l_rope = off; off += (D / 2) * 8;
    a.l_dbg = off;  off += 64;                                        // compute-wave trace stamps
    a.l_end = off;
    return off;
}

// Shapes with a single-launch instantiation: chunks-per-lane of K = H, Hq*D, F
// (K / 2048), head_dim, query heads per kv head and the cache dtype (kvb = 1
// for bf16, 0 for fp16).
bool ps_supported(int cpl_h, int cpl_q, int cpl_f, int D, int gs, int kvb);
// Private-segment (stack/scratch) bytes per lane of the instantiation; the
// single launch is only used when this is zero.
size_t ps_private_bytes(int cpl_h, int cpl_q, int cpl_f, int D, int gs, int kvb);
int ps_slots(int cpl_h, int cpl_q, int cpl_f, int D, int gs, int kvb);   // ring slots per compute wave
// Workgroups of the instantiation that fit on one CU with `lds` bytes of LDS.
int ps_blocks_per_cu(int cpl_h, int cpl_q, int cpl_f, int D, int gs, int kvb, size_t lds);
// coop = true launches through hipLaunchCooperativeKernel, which checks that every
// workgroup is resident at once; coop = false is a plain launch, for which the
// caller has checked that nwg workgroups fit on the device (at most one per CU).
hipError_t launch_persistent(const PsArgs& a, int cpl_h, int cpl_q, int cpl_f, int D, int gs, int kvb, int nwg,
                             size_t lds, bool coop, hipStream_t st);
hipError_t launch_repack_rows(const uint8_t* q, const uint16_t* s, int n, int k, int g, uint8_t* w_out, uint16_t* s_out,
                              int kc, int ng, int row_off, int row_map, int head_dim, hipStream_t st);
hipError_t launch_dequant_rows(const PsMat& m, int kc, int ng, int gchunks, int k, int row_off, int row_map, int n_rows,
                               int head_dim, float* out, hipStream_t st);

// Kernel launchers (kernels.hip).
hipError_t launch_repack(const uint8_t* q, const uint16_t* s, int n, int k, int g,
                         uint8_t* w_out, uint16_t* s_out, int ntiles, int nchunk, int ngroups,
                         int row_off, int row_map, hipStream_t st);
hipError_t launch_gemv(const GemvArgs& a, hipStream_t st);
// Matrix-core product of 1..64 rows (group size 128); a.ksplit splits K.
// Product of 2..64 prepared rows (group size 128); a.ksplit splits K, a.kg groups per wave.
hipError_t launch_gemm_bp(const GemvArgs& a, hipStream_t st);
hipError_t launch_bprep(const void* in, int in_dt, int in_ld, const uint16_t* gamma, int gamma_dt, int K, float eps,
                        int M, uint16_t* bp, float* bc, int kp, float* rs_out, hipStream_t st);
// queries_per_item_max: the largest (rows of an item) x (query heads per kv head).
hipError_t launch_attention(const AttnArgs& a, int head_dim, int queries_per_item_max, hipStream_t st);
hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t v, hipStream_t st);
hipError_t launch_table_gather(const int16_t* src, int16_t* dst, const int* beam, int S, int cap, int P, hipStream_t st);
hipError_t launch_kv_append(uint16_t* kc, uint16_t* vc, int16_t* table, const uint16_t* k, const uint16_t* v,
                            int L, int S, int Hkv, int cap, int D, int P, int n, hipStream_t st);
hipError_t launch_kv_read(const uint16_t* kc, const uint16_t* vc, const int16_t* table, int layer, int slot,
                          int start, int count, int S, int Hkv, int cap, int D, uint16_t* k_out, uint16_t* v_out,
                          hipStream_t st);
hipError_t launch_gemm_pf(const PfArgs& a, hipStream_t st);
// Cache rows P .. P + n - 1 of one layer of a one-slot state (kl, vl: that layer's
// [Hkv][cap][D] base) from n q|k|v result rows: k rotated, both rounded; table
// (layer 0 only, else nullptr) marks the rows as the slot's own.
hipError_t launch_kv_rope_append(const float* qkv, int ld, const int* pos, const float2* rope, int n, int P, int Hq, int Hkv,
                                 int D, uint16_t* kl, uint16_t* vl, int cap, int16_t* table, int kv_dt, hipStream_t st);
// Rows [0, n) of `in` (fp32 or half, row stride in_ld) to 64-row prepared blocks:
// gamma != nullptr: RMSNorm(row) * gamma (full normalization); nullptr: the row as it is.
hipError_t launch_bprep_rows(const void* in, int in_dt, int in_ld, const uint16_t* gamma, int gamma_dt, int K, float eps,
                             int n, uint16_t* bp, float* bc, int kp, hipStream_t st);
hipError_t launch_dequant(const PackedMat& m, int row_off, int row_map, int n_rows, float* out, hipStream_t st);
// Rows src[b][i] (< 0: zero padding) of every slot's logical view, read through
// `table`, to dst [L][S][Hkv][dst_stride][D] rows i < Pn.
hipError_t launch_kv_gather_rows(const uint16_t* kc, const uint16_t* vc, const int16_t* table, const int* src, int L, int S,
                                 int Hkv, int cap, int D, int Pn, int dst_stride, uint16_t* k_dst, uint16_t* v_dst,
                                 hipStream_t st);
// In place: row i of slot b (every layer, kv head, K and V) = the row src[b][i]
// (src[b][i] >= i, ascending per slot; < 0: zero) of the slot's view through
// `table`; rows i < Pn.
hipError_t launch_kv_compact(uint16_t* kc, uint16_t* vc, const int16_t* table, const int* src, int L, int S, int Hkv,
                             int cap, int D, int Pn, hipStream_t st);
hipError_t launch_table_identity(int16_t* table, int S, int cap, int n, hipStream_t st);
// Per row m < M: the largest of the tiles' maxima, its smallest index, and
// 1 / sum over tiles of se * exp(max_t - max) (the softmax probability of it).
hipError_t launch_top1_merge(const float4* part, int M, int ntiles, int32_t* token, float* p, float* logit, hipStream_t st);

// Row m < n of out [n][H] = row ids[m] (device int32) of table [vocab][H]
// (2-byte elements, copied bit for bit); an id outside [0, vocab) gives a zero
// row and sets *err to 1.
hipError_t launch_embed_gather(const uint16_t* table, const int32_t* ids, int n, int vocab, int H, uint16_t* out,
                               unsigned* err, hipStream_t st);

}  // namespace stg
