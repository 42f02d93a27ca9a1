// Host runtime of libstage: validation, weight repack, workspace, KV states,
// metadata staging and the per-layer launch sequence of stage_forward.
#include "stage.h"
#include "common.h"

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

using namespace stg;

// Fixed device staging of kv_capture_noalloc: one copy per GPU the library
// runs on, held until the process ends.  Host code never passes this name to
// a kernel or copy (on the host it is only a stand-in for the symbol): it uses
// the per-device address hipGetSymbolAddress returned at stage creation.
static __device__ __align__(256) uint8_t scratch[STAGE_STATIC_SCRATCH_BYTES];

namespace {

constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
std::array<uint8_t*, SCRATCH_MAX_DEVICES> g_scratch_ptr{};   // address of `scratch` on each device


thread_local std::string g_err;

int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

#define HIP_TRY(expr)                                                                          \
    do {                                                                                       \
        hipError_t e_ = (expr);                                                                \
        if (e_ != hipSuccess) return fail(STAGE_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
    } while (0)

constexpr int META_RING = 4;
constexpr int PF_ROWS = 2048;            // prompt rows per prefill pass (all layers)

// Looks up the address of `scratch` on the current device `dev` once.
int scratch_init(int dev) {
    if (dev < 0 || dev >= SCRATCH_MAX_DEVICES) return fail(STAGE_E_UNSUPPORTED, "device index beyond the static scratch table");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (g_scratch_ptr[dev]) return STAGE_OK;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return fail(STAGE_E_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_ptr[dev] = (uint8_t*)p;
    return STAGE_OK;
}

uint8_t* scratch_ptr(int dev) {
    if (dev < 0 || dev >= SCRATCH_MAX_DEVICES) return nullptr;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    return g_scratch_ptr[dev];
}

struct DevMat {
    PackedMat pm;
    int ksplit = 1, cps = 1;
    int bp_split = 1, bp_kg = 1;   // prepared-operand product: splits of K, groups of 128 k per wave
};

// K split of a prepared-operand product (a function of the matrix only): about
// one workgroup of 4 waves per CU (more splits of K lengthen the last-arrival
// reduction more than they shorten the streaming; 128 to 2048 were measured),
// each wave a range of whole groups.
void bp_plan(DevMat& m) {
    const int ng = m.pm.ngroups, nt = m.pm.ntiles;
    int S = std::max(1, 256 / nt);
    const int kg = std::max(1, (ng + 4 * S - 1) / (4 * S));
    S = (ng + 4 * kg - 1) / (4 * kg);
    m.bp_split = S;
    m.bp_kg = kg;
}

struct LayerDev {
    DevMat qkv, o, gu, d;
    uint16_t* attn_norm = nullptr;
    uint16_t* ffn_norm = nullptr;
};

int dt_code(int stage_dt) { return stage_dt == STAGE_DTYPE_BF16 ? DT_BF16 : DT_F16; }

size_t align16(size_t x) { return (x + 15) & ~(size_t)15; }

}  // namespace

struct Stage {
    StageConfig cfg{};
    int device = 0;
    std::vector<LayerDev> layers;
    std::vector<void*> allocs;
    float2* rope = nullptr;
    float *x = nullptr, *qkv = nullptr, *attn = nullptr, *act = nullptr, *gpart = nullptr, *apart = nullptr, *ssq = nullptr;
    unsigned *gcnt = nullptr, *acnt = nullptr;
    int ntiles_h = 0;
    // prepared inputs of the matrix-core products (2..64 rows), double-buffered
    bool bp_ok = false;
    int kp = 0;                                        // row stride: max K rounded up to 128
    uint16_t* bp[2] = {nullptr, nullptr};              // [MAX_ROWS][kp] codes
    float* bc[2] = {nullptr, nullptr};                 // [MAX_ROWS][kp / 32] corrections
    float* cbf[2] = {nullptr, nullptr};                // [MAX_ROWS] scale each row was prepared with
    float* rsb = nullptr;                              // [MAX_ROWS] rs of the last normalization
    uint8_t* meta_dev = nullptr;
    size_t meta_cap = 0;
    uint8_t* meta_host[META_RING] = {};
    hipEvent_t meta_ev[META_RING] = {};
    bool meta_ev_used[META_RING] = {};
    int ring_i = 0;
    int64_t weight_bytes = 0;
    uint64_t fingerprint = 0;                          // of the config, rotary table and norm weights (KV blobs)
    // final-stage epilogue: final RMSNorm weight and INT4 LM head (stage_head_attach)
    bool head_ok = false;
    int vocab = 0;
    DevMat head;
    uint16_t* final_norm = nullptr;
    float4* top1_part = nullptr;                       // [MAX_ROWS][head tiles]
    // first-stage role: token embedding table [embed_vocab][H] in act dtype (stage_embed_attach)
    uint16_t* embed = nullptr;
    int embed_vocab = 0;
    unsigned* embed_err = nullptr;                     // set by a gather that met an id outside the table
    // prefill workspace for pf_rows prompt rows: residual fp32 [rows][H], q|k|v fp32
    // [rows][NQKV], SwiGLU output fp32 [rows][F], prepared inputs (64-row blocks)
    float *pf_x = nullptr, *pf_qkv = nullptr, *pf_act = nullptr, *pf_bc = nullptr;
    uint16_t* pf_bp = nullptr;
    size_t pf_rows = 0;
    // persistent-kernel weights (row layout) and barrier state
    bool ps_ok = false;
    int cpl_h = 0, cpl_q = 0, cpl_f = 0, kc_h = 0, kc_q = 0, kc_f = 0, ng_h = 0, ng_q = 0, ng_f = 0;
    std::vector<PsLayer> ps_host;
    PsLayer* ps_layers = nullptr;
    uint8_t* ps_wb[4] = {nullptr, nullptr, nullptr, nullptr};   // code slabs per matrix kind (all layers)
    size_t ps_wl[4] = {0, 0, 0, 0};                            // bytes per layer in each slab
    unsigned* err = nullptr;
    unsigned spin_limit = 1u << 20;                     // exchange wait passes (STAGE_PS_SPIN_LIMIT)
    int dbg_layer = -1, dbg_keys = 0, dbg_rows = 0;     // armed attention record (test support)
    float* dbg_q = nullptr;                             // [MAX_ROWS][Hq][D]
    float* dbg_logits = nullptr;                        // [MAX_ROWS][Hq][dbg_keys]
    int ps_nwg = 0;
    int n_cus = 0;                                      // compute units of the device
    int ps_rpw_qkv = 0, ps_rpw_h = 0, ps_rpw_gu = 0;    // rows per workgroup of the single-launch forward
    unsigned long long *ll_qkv = nullptr, *ll_o = nullptr, *ll_part = nullptr, *ll_act = nullptr;   // its flag-word
    unsigned* ll_x = nullptr;                                                                       // exchange buffers
    unsigned ll_epoch = 0;                              // flag numbers used so far
    bool ps_coop = false;                               // cooperative launch (STAGE_COOP=1), else a plain launch
    int attn_vector = 0;                                // attention on the vector units (STAGE_ATTN_VECTOR=1)
    bool attn_dma = true;                               // cache rows by direct loads where allowed (STAGE_ATTN_DMA=0: off)
    int gemm_min_rows = 1;                              // rows from which products use the matrix cores (STAGE_GEMM_MIN_ROWS)
    unsigned long long* trace = nullptr;   // phase stamps of the last persistent forward (STAGE_PS_TRACE=1)
    int prof_class = -1;
    std::vector<hipEvent_t> prof_ev;   // start/stop pairs
    size_t prof_used = 0;              // events recorded
    // Device work of every call on this stage (and on its KV states) runs in call
    // order: done_ev marks the end of the last call's work on last_stream, and a
    // call on another stream waits for it first (see order_on / mark_done).
    hipEvent_t done_ev = nullptr;
    hipStream_t last_stream = nullptr;
    bool done_used = false;

    ~Stage() {
        for (hipEvent_t e : prof_ev) (void)hipEventDestroy(e);
        if (pf_x) {
            (void)hipSetDevice(device);
            (void)hipDeviceSynchronize();
            for (void* p : {(void*)pf_x, (void*)pf_qkv, (void*)pf_act, (void*)pf_bc, (void*)pf_bp}) (void)hipFree(p);
        }
        if (done_ev) (void)hipEventDestroy(done_ev);
        (void)hipSetDevice(device);
        (void)hipDeviceSynchronize();
        for (void* p : allocs) (void)hipFree(p);
        if (meta_dev) (void)hipFree(meta_dev);
        for (int i = 0; i < META_RING; ++i) {
            if (meta_host[i]) (void)hipHostFree(meta_host[i]);
            if (meta_ev[i]) (void)hipEventDestroy(meta_ev[i]);
        }
    }

    template <class T>
    int alloc(T** p, size_t n_elems) {
        void* q = nullptr;
        if (n_elems == 0) n_elems = 1;
        if (hipMalloc(&q, n_elems * sizeof(T)) != hipSuccess) {
            (void)hipGetLastError();
            return fail(STAGE_E_OOM, "device allocation of " + std::to_string(n_elems * sizeof(T)) + " bytes failed");
        }
        allocs.push_back(q);
        *p = (T*)q;
        return STAGE_OK;
    }
};

struct KVState {
    Stage* stage = nullptr;
    int S = 0, cap = 0, P = 0;
    uint16_t* kc = nullptr;
    uint16_t* vc = nullptr;
    int16_t* table[2] = {nullptr, nullptr};
    int cur = 0;
};

namespace {

// Chunks per wave (CPW) of a matrix: the largest of 16, 8, 4, 2, 1 that still
// gives at least `target` workgroups (tiles x K-splits).  K is padded with zero
// codes to a whole number of workgroup slices (4 * CPW chunks each).
int plan_cpw(int ntiles, int nchunk) {
    int target = 1024;
    if (const char* e = std::getenv("STAGE_GEMV_WG_TARGET")) target = std::max(1, atoi(e));
    for (int cpw : {16, 8, 4, 2}) {
        const int cps = 4 * cpw;
        const int nck = (nchunk + cps - 1) / cps * cps;
        if (nck - nchunk > nchunk / 8) continue;           // at most 12.5% padding
        if ((long)ntiles * (nck / cps) >= target) return cpw;
    }
    return 1;
}

int make_mat(Stage* st, DevMat& m, int n_rows_padded_tiles, int k, int g) {
    m.pm.k = k;
    m.pm.ntiles = n_rows_padded_tiles;
    const int nchunk = (k + CHUNK_K - 1) / CHUNK_K;
    const int cpw = plan_cpw(m.pm.ntiles, nchunk);
    m.cps = 4 * cpw;
    m.pm.nchunk = (nchunk + m.cps - 1) / m.cps * m.cps;
    m.ksplit = m.pm.nchunk / m.cps;
    m.pm.gchunks = g / CHUNK_K;
    m.pm.ngroups = (m.pm.nchunk + m.pm.gchunks - 1) / m.pm.gchunks;
    uint8_t* w;
    uint16_t* s;
    const size_t wbytes = (size_t)m.pm.ntiles * m.pm.nchunk * 64 * 16;
    const size_t selems = (size_t)m.pm.ntiles * m.pm.ngroups * 64;
    int rc = st->alloc(&w, wbytes);
    if (rc) return rc;
    rc = st->alloc(&s, selems);
    if (rc) return rc;
    HIP_TRY(hipMemset(w, 0x88, wbytes));
    HIP_TRY(hipMemset(s, 0, selems * sizeof(uint16_t)));
    m.pm.w = w;
    m.pm.s = s;
    st->weight_bytes += (int64_t)wbytes + (int64_t)selems * 2;
    return STAGE_OK;
}

// Copy one canonical matrix into the tiled layout of `m` (rows placed per
// row_off / row_map) and, when `pm` is given, into the row layout as well.
int upload_mat(Stage* st, DevMat& m, const QuantMatrix& q, int on_device, int row_off, int row_map,
               uint8_t* tmp_q, uint16_t* tmp_s, hipStream_t stream, const PsMat* pm = nullptr, int kc = 0, int ng = 0,
               int pm_map = -1) {
    const int g = st->cfg.group_size;
    const size_t qbytes = (size_t)q.n * ((q.k + 1) / 2);
    const size_t sbytes = (size_t)q.n * ((q.k + g - 1) / g) * 2;
    const uint8_t* qsrc = q.q;
    const uint16_t* ssrc = q.scales;
    if (!on_device) {
        HIP_TRY(hipMemcpyAsync(tmp_q, q.q, qbytes, hipMemcpyHostToDevice, stream));
        HIP_TRY(hipMemcpyAsync(tmp_s, q.scales, sbytes, hipMemcpyHostToDevice, stream));
        qsrc = tmp_q;
        ssrc = tmp_s;
    }
    HIP_TRY(launch_repack(qsrc, ssrc, q.n, q.k, g, (uint8_t*)m.pm.w, (uint16_t*)m.pm.s, m.pm.ntiles, m.pm.nchunk,
                          m.pm.ngroups, row_off, row_map, stream));
    if (pm)
        HIP_TRY(launch_repack_rows(qsrc, ssrc, q.n, q.k, g, (uint8_t*)pm->w, (uint16_t*)pm->s, kc, ng, row_off,
                                   pm_map < 0 ? row_map : pm_map, st->cfg.head_dim, stream));
    if (!on_device) HIP_TRY(hipStreamSynchronize(stream));   // tmp buffers are reused by the next matrix
    return STAGE_OK;
}

// Row-layout storage of one matrix kind for all layers: codes in one slab
// (layer l at l * n * kc * 16 bytes), scales in another; padding codes are
// zero (0x88) and the scale slab has a tail so whole 1 KB blocks stay in bounds.
int make_rows(Stage* st, int m, int n_layers, int n, int kc, int ng) {
    uint8_t* w;
    uint16_t* s;
    const size_t wl = (size_t)n * kc * 16, sl = (size_t)n * ng;
    int rc = st->alloc(&w, wl * n_layers);
    if (rc) return rc;
    rc = st->alloc(&s, sl * n_layers + SK_SLOT / 2);
    if (rc) return rc;
    HIP_TRY(hipMemset(w, 0x88, wl * n_layers));
    HIP_TRY(hipMemset(s, 0, (sl * n_layers + SK_SLOT / 2) * 2));
    st->ps_wb[m] = w;
    st->ps_wl[m] = wl;
    for (int l = 0; l < n_layers; ++l) {
        PsLayer& P = st->ps_host[l];
        PsMat& pm = m == 0 ? P.qkv : m == 1 ? P.o : m == 2 ? P.gu : P.d;
        pm.w = w + l * wl;
        pm.s = s + l * sl;
    }
    return STAGE_OK;
}

int check_mat(const QuantMatrix& m, int n, int k, const char* name, int layer) {
    if (!m.q || !m.scales) return fail(STAGE_E_INVALID, std::string(name) + " of layer " + std::to_string(layer) + " is NULL");
    if (m.n != n || m.k != k)
        return fail(STAGE_E_SHAPE, std::string(name) + " of layer " + std::to_string(layer) + " is [" + std::to_string(m.n) +
                                       ", " + std::to_string(m.k) + "], expected [" + std::to_string(n) + ", " +
                                       std::to_string(k) + "]");
    return STAGE_OK;
}

int check_config(const StageConfig* c) {
    if (!c) return fail(STAGE_E_INVALID, "config is NULL");
    if (c->n_layers < 1 || c->hidden < 2 || c->n_q_heads < 1 || c->n_kv_heads < 1 || c->ffn < 2 || c->max_positions < 1)
        return fail(STAGE_E_INVALID, "non-positive dimension in config");
    if (c->hidden % 8 || c->ffn % 8) return fail(STAGE_E_UNSUPPORTED, "hidden and ffn must be multiples of 8");
    if (c->head_dim != 64 && c->head_dim != 128) return fail(STAGE_E_UNSUPPORTED, "head_dim must be 64 or 128");
    if (c->n_q_heads % c->n_kv_heads) return fail(STAGE_E_INVALID, "n_q_heads must be a multiple of n_kv_heads");
    if (c->group_size < 32 || c->group_size % 32) return fail(STAGE_E_UNSUPPORTED, "group_size must be a multiple of 32");
    if ((c->act_dtype != STAGE_DTYPE_F16 && c->act_dtype != STAGE_DTYPE_BF16) ||
        (c->kv_dtype != STAGE_DTYPE_F16 && c->kv_dtype != STAGE_DTYPE_BF16))
        return fail(STAGE_E_INVALID, "act_dtype and kv_dtype must be STAGE_DTYPE_F16 or STAGE_DTYPE_BF16");
    if (!(c->rms_eps > 0.f)) return fail(STAGE_E_INVALID, "rms_eps must be positive");
    if (!c->rope_cos_sin && !(c->rope_theta > 0.0)) return fail(STAGE_E_INVALID, "rope_theta must be positive");
    return STAGE_OK;
}

int ensure_meta(Stage* st, size_t bytes) {
    if (bytes <= st->meta_cap) return STAGE_OK;
    size_t cap = std::max<size_t>(bytes, 2 * st->meta_cap);
    cap = std::max<size_t>(cap, 1 << 16);
    HIP_TRY(hipDeviceSynchronize());   // old buffers may still be read by queued work
    if (st->meta_dev) HIP_TRY(hipFree(st->meta_dev));
    st->meta_dev = nullptr;
    for (int i = 0; i < META_RING; ++i) {
        if (st->meta_host[i]) HIP_TRY(hipHostFree(st->meta_host[i]));
        st->meta_host[i] = nullptr;
        st->meta_ev_used[i] = false;
    }
    if (hipMalloc(&st->meta_dev, cap) != hipSuccess) {
        (void)hipGetLastError();
        st->meta_cap = 0;
        return fail(STAGE_E_OOM, "metadata allocation failed");
    }
    for (int i = 0; i < META_RING; ++i) {
        if (hipHostMalloc(&st->meta_host[i], cap, hipHostMallocDefault) != hipSuccess) {
            (void)hipGetLastError();
            st->meta_cap = 0;
            return fail(STAGE_E_OOM, "pinned metadata allocation failed");
        }
    }
    st->meta_cap = cap;
    return STAGE_OK;
}

// Calls on one stage run on the device in the order they were made, whatever
// streams they are issued on: the workspace, the metadata buffer and the flag
// numbers of the single-launch forward are per stage.  A call on a stream other
// than the previous call's first makes its stream wait for that call's work.
hipError_t order_on(Stage* st, hipStream_t s) {
    if (st->done_used && s != st->last_stream) return hipStreamWaitEvent(s, st->done_ev, 0);
    return hipSuccess;
}
hipError_t mark_done(Stage* st, hipStream_t s) {
    const hipError_t e = hipEventRecord(st->done_ev, s);
    if (e == hipSuccess) {
        st->done_used = true;
        st->last_stream = s;
    }
    return e;
}

constexpr size_t PROF_MAX_LAUNCHES = 65536;

// Records the start (begin = true) or stop event of a profiled launch.
hipError_t prof_mark(Stage* st, int kclass, bool begin, hipStream_t s) {
    if (st->prof_class != kclass) return hipSuccess;
    if (begin && st->prof_used + 2 > 2 * PROF_MAX_LAUNCHES) return hipSuccess;
    if (!begin && (st->prof_used % 2) == 0) return hipSuccess;   // start was not recorded
    if (st->prof_used == st->prof_ev.size()) {
        hipEvent_t e;
        hipError_t err = hipEventCreate(&e);
        if (err != hipSuccess) return err;
        st->prof_ev.push_back(e);
    }
    return hipEventRecord(st->prof_ev[st->prof_used++], s);
}

// FNV-1a, 64 bit.
uint64_t fnv1a(uint64_t h, const void* p, size_t n) {
    const uint8_t* b = (const uint8_t*)p;
    for (size_t i = 0; i < n; ++i) h = (h ^ b[i]) * 0x100000001b3ULL;
    return h;
}

// Copies `bytes` of host data into the next pinned metadata ring slot and from
// there to the device metadata buffer (stream-ordered); *dev is its device copy.
int meta_upload(Stage* st, const void* host, size_t bytes, hipStream_t s, const uint8_t** dev) {
    int rc = ensure_meta(st, std::max<size_t>(bytes, 16));
    if (rc) return rc;
    const int slot_i = st->ring_i;
    st->ring_i = (st->ring_i + 1) % META_RING;
    if (st->meta_ev_used[slot_i]) HIP_TRY(hipEventSynchronize(st->meta_ev[slot_i]));
    if (bytes) std::memcpy(st->meta_host[slot_i], host, bytes);
    HIP_TRY(hipMemcpyAsync(st->meta_dev, st->meta_host[slot_i], std::max<size_t>(bytes, 16), hipMemcpyHostToDevice, s));
    HIP_TRY(hipEventRecord(st->meta_ev[slot_i], s));
    st->meta_ev_used[slot_i] = true;
    *dev = st->meta_dev;
    return STAGE_OK;
}

// Kept rows of every slot: src[b * Pn + i] = the i-th kept row of slot b
// (ascending) or -1 past the slot's count; Pn = the largest count.
void plan_keep(const KVState* kv, const uint8_t* keep, std::vector<int>& src, std::vector<int32_t>& lens, int& Pn) {
    const int S = kv->S, P = kv->P;
    lens.assign(S, 0);
    for (int b = 0; b < S; ++b)
        for (int j = 0; j < P; ++j) lens[b] += (!keep || keep[(size_t)b * P + j]) ? 1 : 0;
    Pn = 0;
    for (int b = 0; b < S; ++b) Pn = std::max(Pn, (int)lens[b]);
    src.assign((size_t)S * Pn, -1);
    for (int b = 0; b < S; ++b) {
        int i = 0;
        for (int j = 0; j < P; ++j)
            if (!keep || keep[(size_t)b * P + j]) src[(size_t)b * Pn + i++] = j;
    }
}

size_t blob_header_bytes(int S) { return (sizeof(StageKVBlobHeader) + 4 * (size_t)S + 255) / 256 * 256; }
size_t blob_rows_bytes(const StageConfig& c, int S, int Pn) {
    return (size_t)c.n_layers * S * c.n_kv_heads * Pn * c.head_dim * 2;   // one of K, V
}

// Header and slot lengths of a capture, zero-padded to header_bytes.
std::vector<uint8_t> blob_header(const Stage* st, int S, int Pn, const std::vector<int32_t>& lens) {
    const StageConfig& c = st->cfg;
    std::vector<uint8_t> h(blob_header_bytes(S), 0);
    StageKVBlobHeader hd{};
    hd.magic = STAGE_KV_BLOB_MAGIC;
    hd.version = STAGE_KV_BLOB_VERSION;
    hd.header_bytes = (uint32_t)h.size();
    hd.fingerprint = st->fingerprint;
    hd.n_layers = c.n_layers;
    hd.n_slots = S;
    hd.n_kv_heads = c.n_kv_heads;
    hd.head_dim = c.head_dim;
    hd.kv_dtype = c.kv_dtype;
    hd.length = Pn;
    std::memcpy(h.data(), &hd, sizeof(hd));
    std::memcpy(h.data() + sizeof(hd), lens.data(), 4 * (size_t)S);
    return h;
}

}  // namespace

// ====================================================================== C ABI

extern "C" {

const char* stage_last_error(void) { return g_err.c_str(); }

int stage_create(const StageConfig* cfg, const LayerWeights* layers, int weights_on_device, void* stream, Stage** out) {
    if (!out) return fail(STAGE_E_INVALID, "out is NULL");
    *out = nullptr;
    int rc = check_config(cfg);
    if (rc) return rc;
    if (!layers) return fail(STAGE_E_INVALID, "layers is NULL");
    const StageConfig& c = *cfg;
    const int H = c.hidden, D = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads, F = c.ffn;
    const int QD = Hq * D, KVD = Hkv * D;
    for (int l = 0; l < c.n_layers; ++l) {
        const LayerWeights& w = layers[l];
        if (!w.attn_norm || !w.ffn_norm) return fail(STAGE_E_INVALID, "norm weight of layer " + std::to_string(l) + " is NULL");
        if ((rc = check_mat(w.wq, QD, H, "wq", l)) || (rc = check_mat(w.wk, KVD, H, "wk", l)) ||
            (rc = check_mat(w.wv, KVD, H, "wv", l)) || (rc = check_mat(w.wo, H, QD, "wo", l)) ||
            (rc = check_mat(w.wg, F, H, "wg", l)) || (rc = check_mat(w.wu, F, H, "wu", l)) ||
            (rc = check_mat(w.wd, H, F, "wd", l)))
            return rc;
    }
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    hipStream_t s = (hipStream_t)stream;

    if (int rc0 = scratch_init(dev)) return rc0;
    Stage* st = new Stage();
    st->cfg = c;
    st->cfg.rope_cos_sin = nullptr;
    st->device = dev;
    st->layers.resize(c.n_layers);

    auto cleanup = [&](int code) {
        delete st;
        return code;
    };

    const int nqkv = QD + 2 * KVD;
    const int g = c.group_size;
    size_t max_q = 0, max_s = 0;
    auto upd = [&](int n, int k) {
        max_q = std::max(max_q, (size_t)n * ((k + 1) / 2));
        max_s = std::max(max_s, (size_t)n * ((k + g - 1) / g));
    };
    upd(QD, H); upd(KVD, H); upd(H, QD); upd(F, H); upd(H, F);
    uint8_t* tmp_q = nullptr;
    uint16_t* tmp_s = nullptr;
    if (!weights_on_device) {
        if (hipMalloc(&tmp_q, max_q) != hipSuccess || hipMalloc(&tmp_s, max_s * 2) != hipSuccess) {
            (void)hipGetLastError();
            if (tmp_q) (void)hipFree(tmp_q);
            return cleanup(fail(STAGE_E_OOM, "staging allocation failed"));
        }
    }
    auto free_tmp = [&]() {
        if (tmp_q) (void)hipFree(tmp_q);
        if (tmp_s) (void)hipFree(tmp_s);
    };

    {
        auto cpl = [](int k) { return (k + PS_KCHUNK - 1) / PS_KCHUNK; };
        st->cpl_h = cpl(H);
        st->cpl_q = cpl(QD);
        st->cpl_f = cpl(F);
        st->kc_h = st->cpl_h * 64;
        st->kc_q = st->cpl_q * 64;
        st->kc_f = st->cpl_f * 64;
        const int gch = g / CHUNK_K;
        st->ng_h = (st->kc_h + gch - 1) / gch;
        st->ng_q = (st->kc_q + gch - 1) / gch;
        st->ng_f = (st->kc_f + gch - 1) / gch;
        const char* e = std::getenv("STAGE_PERSISTENT");
        st->ps_ok = ps_supported(st->cpl_h, st->cpl_q, st->cpl_f, D, Hq / Hkv, c.kv_dtype == STAGE_DTYPE_BF16) &&
                    !(e && atoi(e) == 0);
        if (st->ps_ok) st->ps_host.resize(c.n_layers);
    }
    if (const char* e = std::getenv("STAGE_GEMM_MIN_ROWS")) st->gemm_min_rows = std::max(1, atoi(e));
    if (const char* e = std::getenv("STAGE_ATTN_VECTOR")) st->attn_vector = atoi(e) != 0;
    if (const char* e = std::getenv("STAGE_ATTN_DMA")) st->attn_dma = atoi(e) != 0;
    for (int l = 0; l < c.n_layers; ++l) {
        LayerDev& L = st->layers[l];
        const LayerWeights& w = layers[l];
        PsLayer* P = st->ps_ok ? &st->ps_host[l] : nullptr;
        if (P && l == 0 &&
            ((rc = make_rows(st, 0, c.n_layers, nqkv, st->kc_h, st->ng_h)) ||
             (rc = make_rows(st, 1, c.n_layers, H, st->kc_q, st->ng_q)) ||
             (rc = make_rows(st, 2, c.n_layers, 2 * F, st->kc_h, st->ng_h)) ||
             (rc = make_rows(st, 3, c.n_layers, H, st->kc_f, st->ng_f)))) {
            free_tmp();
            return cleanup(rc);
        }
        if ((rc = make_mat(st, L.qkv, (nqkv + 63) / 64, H, g)) || (rc = make_mat(st, L.o, (H + 63) / 64, QD, g)) ||
            (rc = make_mat(st, L.gu, (F + 31) / 32, H, g)) || (rc = make_mat(st, L.d, (H + 63) / 64, F, g))) {
            free_tmp();
            return cleanup(rc);
        }
        L.qkv.pm.n = nqkv;
        L.o.pm.n = H;
        L.gu.pm.n = 2 * F;
        L.d.pm.n = H;
        const int kh = st->kc_h, kq = st->kc_q, kf = st->kc_f, gh = st->ng_h, gq = st->ng_q, gf = st->ng_f;
        if ((rc = upload_mat(st, L.qkv, w.wq, weights_on_device, 0, 0, tmp_q, tmp_s, s, P ? &P->qkv : nullptr, kh, gh, 3)) ||
            (rc = upload_mat(st, L.qkv, w.wk, weights_on_device, QD, 0, tmp_q, tmp_s, s, P ? &P->qkv : nullptr, kh, gh, 3)) ||
            (rc = upload_mat(st, L.qkv, w.wv, weights_on_device, QD + KVD, 0, tmp_q, tmp_s, s, P ? &P->qkv : nullptr, kh, gh,
                             3)) ||
            (rc = upload_mat(st, L.o, w.wo, weights_on_device, 0, 0, tmp_q, tmp_s, s, P ? &P->o : nullptr, kq, gq)) ||
            (rc = upload_mat(st, L.gu, w.wg, weights_on_device, 0, 1, tmp_q, tmp_s, s, P ? &P->gu : nullptr, kh, gh)) ||
            (rc = upload_mat(st, L.gu, w.wu, weights_on_device, 0, 2, tmp_q, tmp_s, s, P ? &P->gu : nullptr, kh, gh)) ||
            (rc = upload_mat(st, L.d, w.wd, weights_on_device, 0, 0, tmp_q, tmp_s, s, P ? &P->d : nullptr, kf, gf))) {
            free_tmp();
            return cleanup(rc);
        }
        const size_t nalloc = ((size_t)H + SK_SLOT / 2 - 1) / (SK_SLOT / 2) * (SK_SLOT / 2);   // whole 1 KB blocks
        if ((rc = st->alloc(&L.attn_norm, nalloc)) || (rc = st->alloc(&L.ffn_norm, nalloc))) {
            free_tmp();
            return cleanup(rc);
        }
        const hipMemcpyKind kind = weights_on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
        if (hipMemcpyAsync(L.attn_norm, w.attn_norm, (size_t)H * 2, kind, s) != hipSuccess ||
            hipMemcpyAsync(L.ffn_norm, w.ffn_norm, (size_t)H * 2, kind, s) != hipSuccess) {
            free_tmp();
            return cleanup(fail(STAGE_E_HIP, "norm weight copy failed"));
        }
        st->weight_bytes += 4 * (int64_t)H;
        if (P) {
            P->attn_norm = L.attn_norm;
            P->ffn_norm = L.ffn_norm;
        }
    }
    if (hipStreamSynchronize(s) != hipSuccess) {
        free_tmp();
        return cleanup(fail(STAGE_E_HIP, std::string("weight upload: ") + hipGetErrorString(hipGetLastError())));
    }
    free_tmp();

    // rotary table: cos/sin(p * theta^(-2i/D)) in fp64, stored fp32
    const size_t nrope = (size_t)c.max_positions * (D / 2);
    std::vector<float2> rope(nrope);
    if (cfg->rope_cos_sin) {
        for (size_t i = 0; i < nrope; ++i) rope[i] = make_float2(cfg->rope_cos_sin[2 * i], cfg->rope_cos_sin[2 * i + 1]);
    } else {
        for (int p = 0; p < c.max_positions; ++p)
            for (int i = 0; i < D / 2; ++i) {
                const double inv = std::pow(c.rope_theta, -(2.0 * i) / D);
                const double phi = (double)p * inv;
                rope[(size_t)p * (D / 2) + i] = make_float2((float)std::cos(phi), (float)std::sin(phi));
            }
    }
    if ((rc = st->alloc(&st->rope, nrope))) return cleanup(rc);
    if (hipMemcpy(st->rope, rope.data(), nrope * sizeof(float2), hipMemcpyHostToDevice) != hipSuccess)
        return cleanup(fail(STAGE_E_HIP, "rope upload failed"));

    // workspace
    st->ntiles_h = (H + 63) / 64;
    size_t gpart = 0;
    unsigned max_tiles = 0;
    st->bp_ok = true;
    for (auto& L : st->layers)
        for (DevMat* m : {&L.qkv, &L.o, &L.gu, &L.d}) {
            bp_plan(*m);
            st->bp_ok = st->bp_ok && m->pm.gchunks == 4 && m->pm.k % 8 == 0;
            gpart = std::max(gpart, (size_t)m->ksplit * GEMV_MAX_M * m->pm.ntiles * 64);
            gpart = std::max(gpart, (size_t)m->bp_split * MAX_ROWS * m->pm.ntiles * 64);
            max_tiles = std::max<unsigned>(max_tiles, m->pm.ntiles);
        }
    st->kp = (std::max(H, std::max(QD, F)) + 127) / 128 * 128;
    for (int i = 0; i < 2; ++i)
        if ((rc = st->alloc(&st->bp[i], (size_t)MAX_ROWS * st->kp)) || (rc = st->alloc(&st->bc[i], (size_t)MAX_ROWS * st->kp / 32)) ||
            (rc = st->alloc(&st->cbf[i], (size_t)MAX_ROWS)))
            return cleanup(rc);
    if ((rc = st->alloc(&st->rsb, (size_t)MAX_ROWS))) return cleanup(rc);
    for (int i = 0; i < 2; ++i)
        if (hipMemset(st->bp[i], 0, (size_t)MAX_ROWS * st->kp * 2) != hipSuccess ||
            hipMemset(st->bc[i], 0, (size_t)MAX_ROWS * st->kp / 32 * 4) != hipSuccess ||
            hipMemset(st->cbf[i], 0, (size_t)MAX_ROWS * 4) != hipSuccess)
            return cleanup(fail(STAGE_E_HIP, "workspace init failed"));
    if ((rc = st->alloc(&st->x, (size_t)MAX_ROWS * H)) || (rc = st->alloc(&st->qkv, (size_t)MAX_ROWS * nqkv)) ||
        (rc = st->alloc(&st->attn, (size_t)MAX_ROWS * QD)) || (rc = st->alloc(&st->act, (size_t)MAX_ROWS * F)) ||
        (rc = st->alloc(&st->ssq, (size_t)MAX_ROWS * st->ntiles_h)) || (rc = st->alloc(&st->gpart, gpart)) ||
        (rc = st->alloc(&st->apart, (size_t)MAX_ROWS * Hq * ATTN_MAX_SPLITS * (D + 4))) ||
        (rc = st->alloc(&st->gcnt, max_tiles)) || (rc = st->alloc(&st->acnt, (size_t)MAX_ROWS * Hkv)))
        return cleanup(rc);
    if (hipMemset(st->gcnt, 0, max_tiles * sizeof(unsigned)) != hipSuccess ||
        hipMemset(st->acnt, 0, (size_t)MAX_ROWS * Hkv * sizeof(unsigned)) != hipSuccess)
        return cleanup(fail(STAGE_E_HIP, "counter init failed"));
    for (int i = 0; i < META_RING; ++i)
        if (hipEventCreateWithFlags(&st->meta_ev[i], hipEventDisableTiming) != hipSuccess)
            return cleanup(fail(STAGE_E_HIP, "event creation failed"));
    if (hipEventCreateWithFlags(&st->done_ev, hipEventDisableTiming) != hipSuccess)
        return cleanup(fail(STAGE_E_HIP, "event creation failed"));
    if ((rc = ensure_meta(st, 1 << 16))) return cleanup(rc);
    if (hipDeviceGetAttribute(&st->n_cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || st->n_cus < 1)
        return cleanup(fail(STAGE_E_HIP, "CU count query failed"));
    if (st->ps_ok) {
        if ((rc = st->alloc(&st->ps_layers, c.n_layers)) || (rc = st->alloc(&st->err, 4))) return cleanup(rc);
        if (const char* e = std::getenv("STAGE_PS_SPIN_LIMIT")) st->spin_limit = (unsigned)std::max(0, atoi(e));
        if (hipMemcpy(st->ps_layers, st->ps_host.data(), sizeof(PsLayer) * c.n_layers, hipMemcpyHostToDevice) != hipSuccess ||
            hipMemset(st->err, 0, 4) != hipSuccess)
            return cleanup(fail(STAGE_E_HIP, "persistent state init failed"));
        const int cus = st->n_cus;
        // Workgroups (at most one per CU, at most 256): rotary pairs stay in one
        // workgroup (even row counts), gate|up rows come four to a flag word pair
        // (multiples of 4), and every workgroup must own rows of q|k|v, of o/down
        // and of gate|up.  The exchanges have no barriers: a buffer is rewritten
        // only after every workgroup has produced data that depends on having
        // read it, which takes every workgroup producing in every phase.
        auto cdiv = [](int a_, int b_) { return (a_ + b_ - 1) / b_; };
        auto rq_of = [&](int n) { return (cdiv(nqkv, n) + 1) / 2 * 2; };
        auto rh_of = [&](int n) { return cdiv(H, n); };
        auto rg_of = [&](int n) { return (cdiv(2 * F, n) + 3) / 4 * 4; };
        int nwg = std::min(cus, 256);
        while (nwg > 1 && ((nwg - 1) * rq_of(nwg) >= nqkv || (nwg - 1) * rh_of(nwg) >= H || (nwg - 1) * rg_of(nwg) >= 2 * F))
            --nwg;
        st->ps_nwg = nwg;
        st->ps_rpw_qkv = rq_of(nwg);
        st->ps_rpw_h = rh_of(nwg);
        st->ps_rpw_gu = rg_of(nwg);
        if (st->ps_rpw_h > 64) st->ps_ok = false;              // one residual row per control lane
        if (Hkv > nwg) st->ps_ok = false;                      // every kv head needs a workgroup
        if (H % 4 || F % 4 || (Hq * D) % 4) st->ps_ok = false; // flag words are polled four values at a time
        for (long bytes : {(long)st->ps_rpw_qkv * st->ng_h, (long)st->ps_rpw_h * st->ng_q, (long)st->ps_rpw_gu * st->ng_h,
                           (long)st->ps_rpw_h * st->ng_f})
            if ((bytes * 2) % 16 != 0) st->ps_ok = false;      // scale rows are loaded in 16-byte pieces
        PsArgs probe{};
        probe.kc_h = st->kc_h; probe.kc_q = st->kc_q; probe.kc_f = st->kc_f;
        probe.ng_h = st->ng_h; probe.ng_q = st->ng_q; probe.ng_f = st->ng_f;
        probe.rpw_qkv = st->ps_rpw_qkv; probe.rpw_h = st->ps_rpw_h; probe.rpw_gu = st->ps_rpw_gu;
        probe.H = H;
        const int kvb = c.kv_dtype == STAGE_DTYPE_BF16;
        const int slots = ps_slots(st->cpl_h, st->cpl_q, st->cpl_f, D, Hq / Hkv, kvb);
        if (slots <= 0 || ps_layout(probe, slots, D, Hq / Hkv) > 160 * 1024) st->ps_ok = false;
        // flag-word buffers start with flag number 0, which no exchange uses
        const size_t max_split = (size_t)std::max(1, std::min(nwg / Hkv, (Hq / Hkv) * D / 8));
        const size_t n_part = (size_t)Hkv * max_split * (Hq / Hkv) * ps_part_words(D);
        const size_t x_words = (size_t)H + 2 * (size_t)((nwg + 1) & ~1);   // 4-byte words
        if ((rc = st->alloc(&st->ll_qkv, nqkv)) || (rc = st->alloc(&st->ll_o, (size_t)Hq * D / 2)) ||
            (rc = st->alloc(&st->ll_part, n_part)) || (rc = st->alloc(&st->ll_x, x_words)) ||
            (rc = st->alloc(&st->ll_act, (size_t)F / 2)))
            return cleanup(rc);
        if (hipMemset(st->ll_qkv, 0, (size_t)nqkv * 8) != hipSuccess || hipMemset(st->ll_o, 0, (size_t)Hq * D / 2 * 8) != hipSuccess ||
            hipMemset(st->ll_part, 0, n_part * 8) != hipSuccess || hipMemset(st->ll_x, 0, x_words * 4) != hipSuccess ||
            hipMemset(st->ll_act, 0, (size_t)F / 2 * 8) != hipSuccess)
            return cleanup(fail(STAGE_E_HIP, "exchange buffer init failed"));
        if (const char* e = std::getenv("STAGE_COOP")) st->ps_coop = atoi(e) != 0;
        if (const char* e = std::getenv("STAGE_PS_TRACE"))
            if (atoi(e) && (rc = st->alloc(&st->trace, (size_t)nwg * c.n_layers * PS_TRACE_PER_LAYER)))
                return cleanup(rc);
        // the single-launch forward is only used when its kernel needs no private
        // segment (no stack, no scratch spills) for this shape
        if (st->ps_ok && ps_private_bytes(st->cpl_h, st->cpl_q, st->cpl_f, D, Hq / Hkv, kvb) != 0) st->ps_ok = false;
        // Workgroups wait on each other's flag words, so all nwg must be resident at
        // once: nwg <= CUs and one workgroup fits per CU.  The plain launch (default:
        // the cooperative one adds ~17 us per forward on MI355X) relies on this check;
        // a workgroup held back by other work on the device delays the others, and
        // an exchange that never completes ends in STAGE_E_DEVICE, not a hang.
        if (st->ps_ok && (nwg > cus || ps_blocks_per_cu(st->cpl_h, st->cpl_q, st->cpl_f, D, Hq / Hkv, kvb,
                                                        (size_t)ps_layout(probe, slots, D, Hq / Hkv)) < 1))
            st->ps_ok = false;
    }
    if (hipDeviceSynchronize() != hipSuccess) return cleanup(fail(STAGE_E_HIP, "stage_create synchronize failed"));
    {
        // identity of the stage for KV blobs: config, rotary table, norm weights
        uint64_t h = 0xcbf29ce484222325ULL;
        const int32_t dims[] = {c.n_layers, c.hidden, c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn, c.group_size,
                                c.act_dtype, c.kv_dtype, c.max_positions};
        h = fnv1a(h, dims, sizeof(dims));
        h = fnv1a(h, &c.rms_eps, sizeof(c.rms_eps));
        h = fnv1a(h, &c.rope_theta, sizeof(c.rope_theta));
        h = fnv1a(h, rope.data(), rope.size() * sizeof(float2));
        std::vector<uint16_t> nw((size_t)H);
        for (const auto& L : st->layers)
            for (const uint16_t* g : {L.attn_norm, L.ffn_norm}) {
                if (hipMemcpy(nw.data(), g, (size_t)H * 2, hipMemcpyDeviceToHost) != hipSuccess)
                    return cleanup(fail(STAGE_E_HIP, "norm weight read-back failed"));
                h = fnv1a(h, nw.data(), nw.size() * 2);
            }
        st->fingerprint = h;
    }
    *out = st;
    return STAGE_OK;
}

int stage_destroy(Stage* stage) {
    if (!stage) return fail(STAGE_E_INVALID, "stage is NULL");
    delete stage;
    return STAGE_OK;
}

int64_t stage_weight_bytes(const Stage* stage) { return stage ? stage->weight_bytes : -1; }

int stage_debug_attn_arm(Stage* st, int layer, int max_keys) {
    if (!st) return fail(STAGE_E_INVALID, "NULL argument");
    if (layer < 0) {
        st->dbg_layer = -1;
        return STAGE_OK;
    }
    if (layer >= st->cfg.n_layers || max_keys < 1) return fail(STAGE_E_INVALID, "layer or max_keys out of range");
    if (st->attn_vector) return fail(STAGE_E_UNSUPPORTED, "the attention record needs the matrix-core attention");
    HIP_TRY(hipSetDevice(st->device));
    const size_t Hq = (size_t)st->cfg.n_q_heads;
    if (max_keys > st->dbg_keys) {                      // buffers grow only (freed with the stage)
        int rc;
        if ((rc = st->alloc(&st->dbg_q, (size_t)MAX_ROWS * Hq * st->cfg.head_dim)) ||
            (rc = st->alloc(&st->dbg_logits, (size_t)MAX_ROWS * Hq * max_keys)))
            return rc;
        st->dbg_keys = max_keys;
    }
    st->dbg_layer = layer;
    st->dbg_rows = 0;
    return STAGE_OK;
}

int stage_debug_attn_read(Stage* st, float* q_host, float* logits_host, int* rows, int* keys) {
    if (!st || !q_host || !logits_host || !rows || !keys) return fail(STAGE_E_INVALID, "NULL argument");
    if (st->dbg_layer < 0 || st->dbg_rows == 0) return fail(STAGE_E_INVALID, "no armed attention record was taken");
    HIP_TRY(hipSetDevice(st->device));
    HIP_TRY(hipDeviceSynchronize());
    const size_t Hq = (size_t)st->cfg.n_q_heads;
    HIP_TRY(hipMemcpy(q_host, st->dbg_q, (size_t)st->dbg_rows * Hq * st->cfg.head_dim * sizeof(float), hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(logits_host, st->dbg_logits, (size_t)st->dbg_rows * Hq * st->dbg_keys * sizeof(float),
                      hipMemcpyDeviceToHost));
    *rows = st->dbg_rows;
    *keys = st->dbg_keys;
    return STAGE_OK;
}

int stage_device_status(Stage* st) {
    if (!st) return fail(STAGE_E_INVALID, "NULL argument");
    if (!st->err && !st->embed_err) return STAGE_OK;   // nothing on the device can flag this stage
    HIP_TRY(hipSetDevice(st->device));
    HIP_TRY(hipDeviceSynchronize());
    unsigned flag = 0u, eflag = 0u;
    if (st->err) HIP_TRY(hipMemcpy(&flag, st->err, sizeof(unsigned), hipMemcpyDeviceToHost));
    if (st->embed_err) HIP_TRY(hipMemcpy(&eflag, st->embed_err, sizeof(unsigned), hipMemcpyDeviceToHost));
    if (flag) HIP_TRY(hipMemset(st->err, 0, sizeof(unsigned)));
    if (eflag) HIP_TRY(hipMemset(st->embed_err, 0, sizeof(unsigned)));
    if (flag)
        return fail(STAGE_E_DEVICE, "a single-launch forward gave up waiting on another workgroup (was the device "
                                    "shared?); its outputs and appended cache rows are invalid");
    if (eflag)
        return fail(STAGE_E_DEVICE, "stage_embed met a token id outside [0, vocab); the rows of such ids were "
                                    "written as zeros");
    return STAGE_OK;
}

int stage_debug_phase_trace(Stage* stage, uint64_t* out_host, int n, int* n_workgroups) {
    if (!stage || !out_host) return fail(STAGE_E_INVALID, "NULL argument");
    if (!stage->trace) return fail(STAGE_E_UNSUPPORTED, "phase trace is off (set STAGE_PS_TRACE=1 before stage_create)");
    const size_t total = (size_t)stage->ps_nwg * stage->cfg.n_layers * PS_TRACE_PER_LAYER;
    if (n < (long long)total) return fail(STAGE_E_CAPACITY, "trace needs " + std::to_string(total) + " entries");
    HIP_TRY(hipSetDevice(stage->device));
    HIP_TRY(hipMemcpy(out_host, stage->trace, total * 8, hipMemcpyDeviceToHost));
    if (n_workgroups) *n_workgroups = stage->ps_nwg;
    return STAGE_OK;
}

int stage_profile_enable(Stage* stage, int kernel_class) {
    if (!stage) return fail(STAGE_E_INVALID, "stage is NULL");
    if (kernel_class < -1 || kernel_class > STAGE_KERNEL_PERSISTENT) return fail(STAGE_E_INVALID, "unknown kernel class");
    stage->prof_class = kernel_class;
    stage->prof_used = 0;
    return STAGE_OK;
}

int stage_profile_read(Stage* stage, int* launches, double* total_ms) {
    if (!stage || !launches || !total_ms) return fail(STAGE_E_INVALID, "NULL argument");
    *launches = 0;
    *total_ms = 0.0;
    const size_t pairs = stage->prof_used / 2;
    if (pairs) {
        HIP_TRY(hipSetDevice(stage->device));
        HIP_TRY(hipEventSynchronize(stage->prof_ev[2 * pairs - 1]));
        double tot = 0.0;
        for (size_t i = 0; i < pairs; ++i) {
            float ms = 0.f;
            HIP_TRY(hipEventElapsedTime(&ms, stage->prof_ev[2 * i], stage->prof_ev[2 * i + 1]));
            tot += ms;
        }
        *launches = (int)pairs;
        *total_ms = tot;
    }
    stage->prof_used = 0;
    return STAGE_OK;
}

int stage_profile_read_each(Stage* stage, float* ms_out, int capacity, int* launches) {
    if (!stage || !launches || (!ms_out && capacity > 0)) return fail(STAGE_E_INVALID, "NULL argument");
    *launches = 0;
    const size_t pairs = stage->prof_used / 2;
    if (pairs) {
        HIP_TRY(hipSetDevice(stage->device));
        HIP_TRY(hipEventSynchronize(stage->prof_ev[2 * pairs - 1]));
        for (size_t i = 0; i < pairs && (long long)i < capacity; ++i)
            HIP_TRY(hipEventElapsedTime(&ms_out[i], stage->prof_ev[2 * i], stage->prof_ev[2 * i + 1]));
        *launches = (int)pairs;
    }
    stage->prof_used = 0;
    return STAGE_OK;
}

int kv_state_alloc(Stage* stage, int n_slots, int capacity, KVState** out) {
    if (!stage || !out) return fail(STAGE_E_INVALID, "NULL argument");
    *out = nullptr;
    if (n_slots < 1 || capacity < 1) return fail(STAGE_E_INVALID, "n_slots and capacity must be positive");
    if (n_slots > MAX_ROWS) return fail(STAGE_E_CAPACITY, "n_slots exceeds STAGE_MAX_ROWS");
    const StageConfig& c = stage->cfg;
    HIP_TRY(hipSetDevice(stage->device));
    KVState* kv = new KVState();
    kv->stage = stage;
    kv->S = n_slots;
    kv->cap = capacity;
    const size_t elems = (size_t)c.n_layers * n_slots * c.n_kv_heads * capacity * c.head_dim;
    if (hipMalloc(&kv->kc, elems * 2) != hipSuccess || hipMalloc(&kv->vc, elems * 2) != hipSuccess ||
        hipMalloc(&kv->table[0], (size_t)n_slots * capacity * 2) != hipSuccess ||
        hipMalloc(&kv->table[1], (size_t)n_slots * capacity * 2) != hipSuccess) {
        (void)hipGetLastError();
        if (kv->kc) (void)hipFree(kv->kc);
        if (kv->vc) (void)hipFree(kv->vc);
        if (kv->table[0]) (void)hipFree(kv->table[0]);
        delete kv;
        return fail(STAGE_E_OOM, "KV state allocation failed");
    }
    *out = kv;
    return STAGE_OK;
}

int kv_state_free(KVState* kv) {
    if (!kv) return fail(STAGE_E_INVALID, "state is NULL");
    (void)hipSetDevice(kv->stage->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(kv->kc);
    (void)hipFree(kv->vc);
    (void)hipFree(kv->table[0]);
    (void)hipFree(kv->table[1]);
    delete kv;
    return STAGE_OK;
}

int kv_state_reset(KVState* kv) {
    if (!kv) return fail(STAGE_E_INVALID, "state is NULL");
    kv->P = 0;
    return STAGE_OK;
}

int kv_length(const KVState* kv, int* length_out) {
    if (!kv || !length_out) return fail(STAGE_E_INVALID, "NULL argument");
    *length_out = kv->P;
    return STAGE_OK;
}

int kv_truncate(KVState* kv, int new_len) {
    if (!kv) return fail(STAGE_E_INVALID, "state is NULL");
    if (new_len < 0 || new_len > kv->P) return fail(STAGE_E_INVALID, "new_len must be in [0, P]");
    kv->P = new_len;
    return STAGE_OK;
}

int kv_append(KVState* kv, const void* k, const void* v, int n_tokens, int on_device, void* stream) {
    if (!kv || !k || !v) return fail(STAGE_E_INVALID, "NULL argument");
    if (n_tokens < 1) return fail(STAGE_E_INVALID, "n_tokens must be positive");
    if (kv->P + n_tokens > kv->cap) return fail(STAGE_E_CAPACITY, "append exceeds the state's capacity");
    if (on_device && (((uintptr_t)k | (uintptr_t)v) & 15)) return fail(STAGE_E_INVALID, "device rows must be 16-byte aligned");
    Stage* st = kv->stage;
    const StageConfig& c = st->cfg;
    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));
    const size_t bytes = (size_t)c.n_layers * kv->S * c.n_kv_heads * n_tokens * c.head_dim * 2;
    const uint16_t* kd = (const uint16_t*)k;
    const uint16_t* vd = (const uint16_t*)v;
    void* tmp = nullptr;
    if (!on_device) {
        if (hipMalloc(&tmp, 2 * bytes) != hipSuccess) {
            (void)hipGetLastError();
            return fail(STAGE_E_OOM, "staging allocation failed");
        }
        if (hipMemcpyAsync(tmp, k, bytes, hipMemcpyHostToDevice, s) != hipSuccess ||
            hipMemcpyAsync((uint8_t*)tmp + bytes, v, bytes, hipMemcpyHostToDevice, s) != hipSuccess) {
            (void)hipFree(tmp);
            return fail(STAGE_E_HIP, "kv_append upload failed");
        }
        kd = (const uint16_t*)tmp;
        vd = (const uint16_t*)((uint8_t*)tmp + bytes);
    }
    hipError_t e = launch_kv_append(kv->kc, kv->vc, kv->table[kv->cur], kd, vd, c.n_layers, kv->S, c.n_kv_heads, kv->cap,
                                    c.head_dim, kv->P, n_tokens, s);
    if (tmp) {
        hipError_t e2 = hipStreamSynchronize(s);
        (void)hipFree(tmp);
        if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return fail(STAGE_E_HIP, std::string("kv_append: ") + hipGetErrorString(e));
    HIP_TRY(mark_done(st, s));
    kv->P += n_tokens;
    return STAGE_OK;
}

int kv_read(KVState* kv, int layer, int slot, int start, int count, void* k_out, void* v_out, int out_on_device,
            void* stream) {
    if (!kv || !k_out || !v_out) return fail(STAGE_E_INVALID, "NULL argument");
    Stage* st = kv->stage;
    const StageConfig& c = st->cfg;
    if (layer < 0 || layer >= c.n_layers || slot < 0 || slot >= kv->S) return fail(STAGE_E_INVALID, "layer or slot out of range");
    if (start < 0 || count < 0 || start + count > kv->P) return fail(STAGE_E_INVALID, "row range exceeds P");
    if (count == 0) return STAGE_OK;
    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));
    const size_t bytes = (size_t)c.n_kv_heads * count * c.head_dim * 2;
    uint16_t* kd = (uint16_t*)k_out;
    uint16_t* vd = (uint16_t*)v_out;
    void* tmp = nullptr;
    if (!out_on_device) {
        if (hipMalloc(&tmp, 2 * bytes) != hipSuccess) {
            (void)hipGetLastError();
            return fail(STAGE_E_OOM, "staging allocation failed");
        }
        kd = (uint16_t*)tmp;
        vd = (uint16_t*)((uint8_t*)tmp + bytes);
    }
    hipError_t e = launch_kv_read(kv->kc, kv->vc, kv->table[kv->cur], layer, slot, start, count, kv->S, c.n_kv_heads,
                                  kv->cap, c.head_dim, kd, vd, s);
    if (tmp) {
        if (e == hipSuccess) e = hipMemcpyAsync(k_out, kd, bytes, hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipMemcpyAsync(v_out, vd, bytes, hipMemcpyDeviceToHost, s);
        hipError_t e2 = hipStreamSynchronize(s);
        (void)hipFree(tmp);
        if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return fail(STAGE_E_HIP, std::string("kv_read: ") + hipGetErrorString(e));
    HIP_TRY(mark_done(st, s));
    return STAGE_OK;
}

int kv_compact(KVState* kv, const uint8_t* keep_mask, int32_t* slot_lengths, void* stream) {
    if (!kv) return fail(STAGE_E_INVALID, "state is NULL");
    Stage* st = kv->stage;
    const StageConfig& c = st->cfg;
    std::vector<int> src;
    std::vector<int32_t> lens;
    int Pn = 0;
    plan_keep(kv, keep_mask, src, lens, Pn);
    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));
    if (Pn > 0) {
        const uint8_t* d = nullptr;
        int rc = meta_upload(st, src.data(), src.size() * sizeof(int), s, &d);
        if (rc) return rc;
        HIP_TRY(launch_kv_compact(kv->kc, kv->vc, kv->table[kv->cur], (const int*)d, c.n_layers, kv->S, c.n_kv_heads,
                                  kv->cap, c.head_dim, Pn, s));
        HIP_TRY(launch_table_identity(kv->table[kv->cur], kv->S, kv->cap, Pn, s));
    }
    HIP_TRY(mark_done(st, s));
    kv->P = Pn;
    if (slot_lengths) std::memcpy(slot_lengths, lens.data(), 4 * (size_t)kv->S);
    return STAGE_OK;
}

int kv_capture_size(const KVState* kv, const uint8_t* keep_mask, int64_t* bytes_out) {
    if (!kv || !bytes_out) return fail(STAGE_E_INVALID, "NULL argument");
    std::vector<int> src;
    std::vector<int32_t> lens;
    int Pn = 0;
    plan_keep(kv, keep_mask, src, lens, Pn);
    *bytes_out = (int64_t)(blob_header_bytes(kv->S) + 2 * blob_rows_bytes(kv->stage->cfg, kv->S, Pn));
    return STAGE_OK;
}

int kv_capture(KVState* kv, const uint8_t* keep_mask, void* blob, int64_t blob_bytes, int blob_on_device, void* stream) {
    if (!kv || !blob) return fail(STAGE_E_INVALID, "NULL argument");
    Stage* st = kv->stage;
    const StageConfig& c = st->cfg;
    std::vector<int> src;
    std::vector<int32_t> lens;
    int Pn = 0;
    plan_keep(kv, keep_mask, src, lens, Pn);
    const std::vector<uint8_t> hdr = blob_header(st, kv->S, Pn, lens);
    const size_t rows = blob_rows_bytes(c, kv->S, Pn);
    if (blob_bytes < 0 || (size_t)blob_bytes < hdr.size() + 2 * rows)
        return fail(STAGE_E_CAPACITY, "blob smaller than kv_capture_size");
    if (blob_on_device && ((uintptr_t)blob & 15)) return fail(STAGE_E_INVALID, "device blob must be 16-byte aligned");
    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));
    // metadata slot: kept-row lists, then the header (copied to a device blob from there)
    const size_t src_bytes = (src.size() * sizeof(int) + 255) / 256 * 256;
    std::vector<uint8_t> meta(src_bytes + hdr.size(), 0);
    std::memcpy(meta.data(), src.data(), src.size() * sizeof(int));
    std::memcpy(meta.data() + src_bytes, hdr.data(), hdr.size());
    const uint8_t* d = nullptr;
    int rc = meta_upload(st, meta.data(), meta.size(), s, &d);
    if (rc) return rc;
    uint8_t* rows_dst = (uint8_t*)blob + hdr.size();   // K rows, then V rows
    void* tmp = nullptr;
    if (!blob_on_device) {
        if (rows && hipMalloc(&tmp, 2 * rows) != hipSuccess) {
            (void)hipGetLastError();
            return fail(STAGE_E_OOM, "capture staging allocation failed");
        }
        rows_dst = (uint8_t*)tmp;
    } else {
        HIP_TRY(hipMemcpyAsync(blob, d + src_bytes, hdr.size(), hipMemcpyDeviceToDevice, s));
    }
    hipError_t e = hipSuccess;
    if (rows)
        e = launch_kv_gather_rows(kv->kc, kv->vc, kv->table[kv->cur], (const int*)d, c.n_layers, kv->S, c.n_kv_heads,
                                  kv->cap, c.head_dim, Pn, Pn, (uint16_t*)rows_dst, (uint16_t*)(rows_dst + rows), s);
    if (!blob_on_device) {
        std::memcpy(blob, hdr.data(), hdr.size());
        if (e == hipSuccess && rows) e = hipMemcpyAsync((uint8_t*)blob + hdr.size(), tmp, 2 * rows, hipMemcpyDeviceToHost, s);
        const hipError_t e2 = hipStreamSynchronize(s);
        if (tmp) (void)hipFree(tmp);
        if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return fail(STAGE_E_HIP, std::string("kv_capture: ") + hipGetErrorString(e));
    HIP_TRY(mark_done(st, s));
    return STAGE_OK;
}

int kv_capture_noalloc(KVState* kv, const uint8_t* keep_mask, void* blob_host, int64_t blob_bytes, void* stream) {
    if (!kv || !blob_host) return fail(STAGE_E_INVALID, "NULL argument");
    Stage* st = kv->stage;
    const StageConfig& c = st->cfg;
    std::vector<int> src;
    std::vector<int32_t> lens;
    int Pn = 0;
    plan_keep(kv, keep_mask, src, lens, Pn);
    const std::vector<uint8_t> hdr = blob_header(st, kv->S, Pn, lens);
    const size_t rows = blob_rows_bytes(c, kv->S, Pn);
    if (blob_bytes < 0 || (size_t)blob_bytes < hdr.size() + 2 * rows)
        return fail(STAGE_E_CAPACITY, "blob smaller than kv_capture_size");
    const size_t src_bytes = (src.size() * sizeof(int) + 255) / 256 * 256;
    const size_t layer_rows = rows / (size_t)c.n_layers;    // one layer's K (or V) rows
    const size_t room = STAGE_STATIC_SCRATCH_BYTES > src_bytes ? STAGE_STATIC_SCRATCH_BYTES - src_bytes : 0;
    const int per = layer_rows ? (int)std::min<size_t>((size_t)c.n_layers, room / (2 * layer_rows)) : c.n_layers;
    if (src_bytes > STAGE_STATIC_SCRATCH_BYTES || per < 1)
        return fail(STAGE_E_CAPACITY, "one layer's kept rows (" + std::to_string(2 * layer_rows) + " bytes) and row lists (" +
                                          std::to_string(src_bytes) + " bytes) exceed STAGE_STATIC_SCRATCH_BYTES");
    HIP_TRY(hipSetDevice(st->device));
    uint8_t* sp = scratch_ptr(st->device);
    if (!sp) return fail(STAGE_E_HIP, "static scratch address unknown on this device");
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));
    std::memcpy(blob_host, hdr.data(), hdr.size());
    uint8_t* kdst = (uint8_t*)blob_host + hdr.size();
    uint8_t* vdst = kdst + rows;
    if (rows) {
        HIP_TRY(hipMemcpyAsync(sp, src.data(), src.size() * sizeof(int), hipMemcpyHostToDevice, s));
        const size_t layer_elems = (size_t)kv->S * c.n_kv_heads * kv->cap * c.head_dim;
        for (int l0 = 0; l0 < c.n_layers; l0 += per) {
            const int nl = std::min(per, c.n_layers - l0);
            uint8_t* ks = sp + src_bytes;
            uint8_t* vs = ks + (size_t)nl * layer_rows;
            HIP_TRY(launch_kv_gather_rows(kv->kc + (size_t)l0 * layer_elems, kv->vc + (size_t)l0 * layer_elems,
                                          kv->table[kv->cur], (const int*)sp, nl, kv->S, c.n_kv_heads, kv->cap, c.head_dim,
                                          Pn, Pn, (uint16_t*)ks, (uint16_t*)vs, s));
            HIP_TRY(hipMemcpyAsync(kdst + (size_t)l0 * layer_rows, ks, (size_t)nl * layer_rows, hipMemcpyDeviceToHost, s));
            HIP_TRY(hipMemcpyAsync(vdst + (size_t)l0 * layer_rows, vs, (size_t)nl * layer_rows, hipMemcpyDeviceToHost, s));
        }
    }
    HIP_TRY(hipStreamSynchronize(s));
    HIP_TRY(mark_done(st, s));
    return STAGE_OK;
}

int kv_restore(KVState* kv, const void* blob, int64_t blob_bytes, int blob_on_device, int32_t* slot_lengths, void* stream) {
    if (!kv || !blob) return fail(STAGE_E_INVALID, "NULL argument");
    Stage* st = kv->stage;
    const StageConfig& c = st->cfg;
    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    if ((size_t)std::max<int64_t>(blob_bytes, 0) < sizeof(StageKVBlobHeader))
        return fail(STAGE_E_SHAPE, "blob shorter than its header");
    if (blob_on_device && ((uintptr_t)blob & 15)) return fail(STAGE_E_INVALID, "device blob must be 16-byte aligned");
    StageKVBlobHeader hd{};
    std::vector<int32_t> lens;
    if (blob_on_device) {
        HIP_TRY(order_on(st, s));
        HIP_TRY(hipMemcpyAsync(&hd, blob, sizeof(hd), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
    } else {
        std::memcpy(&hd, blob, sizeof(hd));
    }
    if (hd.magic != STAGE_KV_BLOB_MAGIC || hd.version != STAGE_KV_BLOB_VERSION)
        return fail(STAGE_E_INVALID, "not a KV blob of this version");
    if (hd.fingerprint != st->fingerprint || hd.n_layers != c.n_layers || hd.n_kv_heads != c.n_kv_heads ||
        hd.head_dim != c.head_dim || hd.kv_dtype != c.kv_dtype)
        return fail(STAGE_E_STATE_MISMATCH, "blob was captured by a different stage");
    if (hd.n_slots != kv->S) return fail(STAGE_E_STATE_MISMATCH, "blob slot count differs from the state's");
    const int S = kv->S, Pn = hd.length;
    if (Pn < 0 || hd.header_bytes != blob_header_bytes(S)) return fail(STAGE_E_SHAPE, "malformed blob header");
    const size_t rows = blob_rows_bytes(c, S, Pn);
    if ((size_t)blob_bytes < hd.header_bytes + 2 * rows) return fail(STAGE_E_SHAPE, "blob shorter than its rows");
    if (Pn > kv->cap) return fail(STAGE_E_CAPACITY, "blob length exceeds the state's capacity");
    lens.resize(S);
    if (blob_on_device) {
        HIP_TRY(hipMemcpy(lens.data(), (const uint8_t*)blob + sizeof(hd), 4 * (size_t)S, hipMemcpyDeviceToHost));
    } else {
        std::memcpy(lens.data(), (const uint8_t*)blob + sizeof(hd), 4 * (size_t)S);
    }
    for (int b = 0; b < S; ++b)
        if (lens[b] < 0 || lens[b] > Pn) return fail(STAGE_E_SHAPE, "malformed slot length in blob");
    HIP_TRY(order_on(st, s));
    const uint16_t* kd = (const uint16_t*)((const uint8_t*)blob + hd.header_bytes);
    void* tmp = nullptr;
    if (!blob_on_device && rows) {
        if (hipMalloc(&tmp, 2 * rows) != hipSuccess) {
            (void)hipGetLastError();
            return fail(STAGE_E_OOM, "restore staging allocation failed");
        }
        if (hipMemcpyAsync(tmp, kd, 2 * rows, hipMemcpyHostToDevice, s) != hipSuccess) {
            (void)hipFree(tmp);
            return fail(STAGE_E_HIP, "restore upload failed");
        }
        kd = (const uint16_t*)tmp;
    }
    hipError_t e = hipSuccess;
    if (Pn > 0)
        e = launch_kv_append(kv->kc, kv->vc, kv->table[kv->cur], kd, (const uint16_t*)((const uint8_t*)kd + rows), c.n_layers,
                             S, c.n_kv_heads, kv->cap, c.head_dim, 0, Pn, s);
    if (tmp) {
        const hipError_t e2 = hipStreamSynchronize(s);
        (void)hipFree(tmp);
        if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return fail(STAGE_E_HIP, std::string("kv_restore: ") + hipGetErrorString(e));
    HIP_TRY(mark_done(st, s));
    kv->P = Pn;
    if (slot_lengths) std::memcpy(slot_lengths, lens.data(), 4 * (size_t)S);
    return STAGE_OK;
}

int stage_head_attach(Stage* st, const uint16_t* final_norm, const QuantMatrix* lm_head, int weights_on_device, void* stream) {
    if (!st || !final_norm || !lm_head || !lm_head->q || !lm_head->scales) return fail(STAGE_E_INVALID, "NULL argument");
    if (st->head_ok) return fail(STAGE_E_UNSUPPORTED, "the stage already has a head");
    const StageConfig& c = st->cfg;
    const int H = c.hidden;
    if (lm_head->n < 1 || lm_head->k != H) return fail(STAGE_E_SHAPE, "lm_head must be [vocab >= 1, hidden]");
    if (!st->bp_ok) return fail(STAGE_E_UNSUPPORTED, "the head needs 128-wide quantization groups");
    if (lm_head->n > (1 << 30)) return fail(STAGE_E_CAPACITY, "vocab too large");
    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));
    const int V = lm_head->n, g = c.group_size;
    DevMat m{};
    int rc = make_mat(st, m, (V + 63) / 64, H, g);
    if (rc) return rc;
    m.pm.n = V;
    // no split of K: the epilogue's per-tile maxima need a tile's whole sums
    m.bp_split = 1;
    m.bp_kg = (m.pm.ngroups + 3) / 4;
    uint8_t* tmp_q = nullptr;
    uint16_t* tmp_s = nullptr;
    if (!weights_on_device) {
        const size_t qbytes = (size_t)V * ((H + 1) / 2), sbytes = (size_t)V * ((H + g - 1) / g) * 2;
        if (hipMalloc(&tmp_q, qbytes) != hipSuccess || hipMalloc(&tmp_s, sbytes) != hipSuccess) {
            (void)hipGetLastError();
            if (tmp_q) (void)hipFree(tmp_q);
            return fail(STAGE_E_OOM, "head upload staging allocation failed");
        }
    }
    rc = upload_mat(st, m, *lm_head, weights_on_device, 0, 0, tmp_q, tmp_s, s);
    if (tmp_q) (void)hipFree(tmp_q);
    if (tmp_s) (void)hipFree(tmp_s);
    if (rc) return rc;
    uint16_t* fn = nullptr;
    float4* part = nullptr;
    const size_t nalloc = ((size_t)H + SK_SLOT / 2 - 1) / (SK_SLOT / 2) * (SK_SLOT / 2);
    if ((rc = st->alloc(&fn, nalloc)) || (rc = st->alloc(&part, (size_t)MAX_ROWS * m.pm.ntiles))) return rc;
    HIP_TRY(hipMemcpyAsync(fn, final_norm, (size_t)H * 2, weights_on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice, s));
    HIP_TRY(hipStreamSynchronize(s));
    st->weight_bytes += 2 * (int64_t)H;
    st->head = m;
    st->final_norm = fn;
    st->top1_part = part;
    st->vocab = V;
    st->head_ok = true;
    HIP_TRY(mark_done(st, s));
    return STAGE_OK;
}

int stage_embed_attach(Stage* st, const uint16_t* table, int vocab, int weights_on_device, void* stream) {
    if (!st || !table) return fail(STAGE_E_INVALID, "NULL argument");
    if (st->embed) return fail(STAGE_E_UNSUPPORTED, "the stage already has an embedding table");
    if (vocab < 1) return fail(STAGE_E_SHAPE, "vocab must be >= 1");
    const int H = st->cfg.hidden;
    if ((int64_t)vocab * H > ((int64_t)1 << 36)) return fail(STAGE_E_CAPACITY, "embedding table too large");
    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));
    uint16_t* t = nullptr;
    unsigned* e = nullptr;
    int rc;
    if ((rc = st->alloc(&t, (size_t)vocab * H)) || (rc = st->alloc(&e, 1))) return rc;
    HIP_TRY(hipMemsetAsync(e, 0, sizeof(unsigned), s));
    HIP_TRY(hipMemcpyAsync(t, table, (size_t)vocab * H * 2, weights_on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice,
                           s));
    HIP_TRY(hipStreamSynchronize(s));
    st->weight_bytes += 2 * (int64_t)vocab * H;
    st->embed = t;
    st->embed_err = e;
    st->embed_vocab = vocab;
    HIP_TRY(mark_done(st, s));
    return STAGE_OK;
}

int stage_embed(Stage* st, const int32_t* ids, int n, void* hidden_out, void* stream) {
    if (!st || !ids || !hidden_out) return fail(STAGE_E_INVALID, "NULL argument");
    if (!st->embed) return fail(STAGE_E_INVALID, "no embedding table attached (stage_embed_attach)");
    if (n < 1 || n > STAGE_MAX_PREFILL) return fail(STAGE_E_CAPACITY, "n must be in [1, STAGE_MAX_PREFILL]");
    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));
    HIP_TRY(launch_embed_gather(st->embed, ids, n, st->embed_vocab, st->cfg.hidden, (uint16_t*)hidden_out, st->embed_err,
                                s));
    HIP_TRY(mark_done(st, s));
    return STAGE_OK;
}

int stage_head_top1(Stage* st, const void* hidden, int M, int32_t* token_out, float* p_out, float* logit_out,
                    float* logits_out, void* stream) {
    if (!st || !hidden || !token_out || !p_out) return fail(STAGE_E_INVALID, "NULL argument");
    if (!st->head_ok) return fail(STAGE_E_INVALID, "no head attached (stage_head_attach)");
    if (M < 1 || M > MAX_ROWS) return fail(STAGE_E_CAPACITY, "M must be in [1, STAGE_MAX_ROWS]");
    const StageConfig& c = st->cfg;
    const int H = c.hidden, act_dt = dt_code(c.act_dtype);
    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));
    HIP_TRY(launch_bprep(hidden, act_dt, H, st->final_norm, act_dt, H, c.rms_eps, M, st->bp[0], st->bc[0], st->kp,
                         st->rsb, s));
    GemvArgs a{};
    a.W = st->head.pm;
    a.M = M;
    a.kp = st->kp;
    a.kg = st->head.bp_kg;
    a.ksplit = 1;
    a.partial = st->gpart;
    a.counters = st->gcnt;
    a.bp_in = st->bp[0];
    a.bc_in = st->bc[0];
    a.cb_in = st->cbf[0];
    a.norm = 2;
    a.epi = EPI_TOP1;
    a.out = logits_out;
    a.out_ld = st->vocab;
    a.top1_part = st->top1_part;
    HIP_TRY(launch_gemm_bp(a, s));
    HIP_TRY(launch_top1_merge(st->top1_part, M, st->head.pm.ntiles, token_out, p_out, logit_out, s));
    HIP_TRY(mark_done(st, s));
    return STAGE_OK;
}

int stage_prefill(Stage* st, KVState* kv, int n, const int32_t* positions, const uint8_t* past_mask, const void* hidden_in,
                  void* hidden_out, void* stream) {
    if (!st || !kv || !positions || !hidden_in || !hidden_out) return fail(STAGE_E_INVALID, "NULL argument");
    if (kv->stage != st) return fail(STAGE_E_STATE_MISMATCH, "state belongs to another stage");
    if (kv->S != 1) return fail(STAGE_E_SHAPE, "prefill takes a one-slot state");
    if (n < 1 || n > STAGE_MAX_PREFILL) return fail(STAGE_E_CAPACITY, "n_tokens must be in [1, STAGE_MAX_PREFILL]");
    if (!st->bp_ok) return fail(STAGE_E_UNSUPPORTED, "prefill needs 128-wide quantization groups");
    const StageConfig& c = st->cfg;
    const int H = c.hidden, D = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads, F = c.ffn;
    const int P0 = kv->P;
    if (P0 + n > kv->cap) return fail(STAGE_E_CAPACITY, "P + n_tokens exceeds the state's capacity");
    for (int i = 0; i < n; ++i)
        if (positions[i] < 0 || positions[i] >= c.max_positions)
            return fail(STAGE_E_CAPACITY, "position " + std::to_string(positions[i]) + " outside the rotary table");
    const int act_dt = dt_code(c.act_dtype), nqkv = Hq * D + 2 * Hkv * D;
    const size_t row_bytes = (size_t)H * 2;
    if ((const uint8_t*)hidden_in < (const uint8_t*)hidden_out + (size_t)n * row_bytes &&
        (const uint8_t*)hidden_out < (const uint8_t*)hidden_in + (size_t)n * row_bytes)
        return fail(STAGE_E_INVALID, "hidden_in and hidden_out overlap");
    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));
    // workspace for one pass of at most PF_ROWS rows
    const int pass_rows = std::min(n, PF_ROWS);
    const size_t wrows = (size_t)(pass_rows + 63) / 64 * 64;
    if (st->pf_rows < wrows) {
        HIP_TRY(hipDeviceSynchronize());
        for (void* p : {(void*)st->pf_x, (void*)st->pf_qkv, (void*)st->pf_act, (void*)st->pf_bc, (void*)st->pf_bp})
            if (p) HIP_TRY(hipFree(p));
        st->pf_x = st->pf_qkv = st->pf_act = st->pf_bc = nullptr;
        st->pf_bp = nullptr;
        st->pf_rows = 0;
        if (hipMalloc(&st->pf_x, wrows * H * 4) != hipSuccess || hipMalloc(&st->pf_qkv, wrows * nqkv * 4) != hipSuccess ||
            hipMalloc(&st->pf_act, wrows * std::max(F, Hq * D) * 4) != hipSuccess ||
            hipMalloc(&st->pf_bp, wrows * st->kp * 2) != hipSuccess ||
            hipMalloc(&st->pf_bc, wrows / 64 * 2 * st->kp * 4) != hipSuccess) {
            (void)hipGetLastError();
            return fail(STAGE_E_OOM, "prefill workspace allocation failed");
        }
        st->pf_rows = wrows;
    }

    // ---------------- one request record per chunk of at most PF_ATT_ROWS rows (the
    // attention's unit), in one upload: chunk q covers prompt rows [16 q, 16 q + m),
    // sees the past rows the mask keeps, the earlier chunks' rows and its own rows
    // causally.  Row numbers (row0, positions, row_item) count from the start of
    // the chunk's pass.  16-row chunks keep a chunk's query vectors (16 x query
    // heads per kv head) within one or two tiles per wave, so the attention runs
    // two workgroups per CU without spilling; the chunks of one context read the
    // same cache rows, mostly from the caches.
    constexpr int PF_ATT_ROWS = 16;
    const int nch = (n + PF_ATT_ROWS - 1) / PF_ATT_ROWS;
    const int pass_chunks = PF_ROWS / PF_ATT_ROWS;
    size_t mask_total = 0;
    for (int q = 0; q < nch; ++q)
        mask_total += (size_t)P0 + q * PF_ATT_ROWS + std::min(PF_ATT_ROWS, n - q * PF_ATT_ROWS);
    const size_t off_req = 0;
    const size_t off_item = align16(off_req + sizeof(ReqDev) * nch);
    const size_t off_pos = align16(off_item + sizeof(ItemDev) * nch);
    const size_t off_ritem = align16(off_pos + sizeof(int) * n);
    const size_t off_mask = align16(off_ritem + sizeof(int) * n);
    const size_t total = align16(off_mask + mask_total);
    int rc = ensure_meta(st, total);
    if (rc) return rc;
    const int slot_i = st->ring_i;
    st->ring_i = (st->ring_i + 1) % META_RING;
    if (st->meta_ev_used[slot_i]) HIP_TRY(hipEventSynchronize(st->meta_ev[slot_i]));
    uint8_t* hb = st->meta_host[slot_i];
    const int splits = 2;                              // per (chunk, kv head): the chunks fill the device
    {
        size_t moff = 0;
        for (int q = 0; q < nch; ++q) {
            const int r0 = q * PF_ATT_ROWS, m = std::min(PF_ATT_ROWS, n - r0);
            const int qf = q / pass_chunks * pass_chunks;   // first chunk of the pass
            ReqDev d{};
            d.P = P0 + r0;
            d.n = m;
            d.S = 1;
            d.row0 = (q - qf) * PF_ATT_ROWS;
            d.cap = kv->cap;
            d.mask_off = (int)moff;
            d.mask_len = P0 + r0 + m;
            d.rowmask_off = -1;
            d.item0 = q - qf;
            d.splits = splits;
            d.kc = kv->kc;
            d.vc = kv->vc;
            d.table = kv->table[kv->cur];
            ((ReqDev*)(hb + off_req))[q] = d;
            ((ItemDev*)(hb + off_item))[q] = ItemDev{q - qf, 0, d};
            for (int i = 0; i < m; ++i) ((int*)(hb + off_ritem))[r0 + i] = q - qf;
            uint8_t* mk = hb + off_mask + moff;
            for (int jj = 0; jj < P0; ++jj) mk[jj] = past_mask ? (past_mask[jj] ? 1 : 0) : 1;
            std::memset(mk + P0, 1, (size_t)r0 + m);
            moff += (size_t)P0 + r0 + m;
        }
        std::memcpy(hb + off_pos, positions, sizeof(int) * n);
    }
    uint8_t* db = st->meta_dev;
    HIP_TRY(hipMemcpyAsync(db, hb, total, hipMemcpyHostToDevice, s));
    HIP_TRY(hipEventRecord(st->meta_ev[slot_i], s));
    st->meta_ev_used[slot_i] = true;
    if ((size_t)PF_ROWS * Hq * splits * (D + 2) > (size_t)MAX_ROWS * Hq * ATTN_MAX_SPLITS * (D + 4))
        return fail(STAGE_E_UNSUPPORTED, "attention partials of a prefill pass exceed the workspace");

    // ---------------- passes of at most PF_ROWS rows, each through every layer: the
    // products take all of a pass's rows at once (gemm_pf_kernel), the attention
    // one 64-row chunk at a time (its keys include the earlier chunks' rows)
    const int kp = st->kp;
    const size_t bp_blk = (size_t)64 * kp, bc_blk = (size_t)2 * kp;
    auto pf = [&](const DevMat& mat, int rows, int epi) {
        PfArgs a{};
        a.W = mat.pm;
        a.bp = st->pf_bp;
        a.bc = st->pf_bc;
        a.bp_blk = bp_blk;
        a.bc_blk = bc_blk;
        a.n = rows;
        a.epi = epi;
        a.nwt = (mat.pm.ntiles + 3) / 4;
        a.ntb = (rows + 63) / 64;
        return a;
    };
    for (int p0 = 0; p0 < n; p0 += PF_ROWS) {
        const int pr = std::min(PF_ROWS, n - p0);
        const uint8_t* hin = (const uint8_t*)hidden_in + (size_t)p0 * row_bytes;
        for (int l = 0; l < c.n_layers; ++l) {
            const LayerDev& Ld = st->layers[l];
            const bool first = (l == 0), last = (l == c.n_layers - 1);
            // q|k|v = RMSNorm(x) W_qkv^T
            HIP_TRY(prof_mark(st, STAGE_KERNEL_QKV, true, s));
            HIP_TRY(launch_bprep_rows(first ? (const void*)hin : (const void*)st->pf_x, first ? act_dt : DT_F32, H,
                                      Ld.attn_norm, act_dt, H, c.rms_eps, pr, st->pf_bp, st->pf_bc, kp, s));
            {
                PfArgs a = pf(Ld.qkv, pr, EPI_STORE);
                a.out = st->pf_qkv;
                a.out_ld = nqkv;
                HIP_TRY(launch_gemm_pf(a, s));
            }
            HIP_TRY(prof_mark(st, STAGE_KERNEL_QKV, false, s));
            // the pass's k and v rows into the cache, then the causal attention of all its
            // 16-row chunks in one launch (each a request whose past includes the
            // earlier chunks' rows); the output goes to the o product as prepared blocks
            HIP_TRY(prof_mark(st, STAGE_KERNEL_ATTN, true, s));
            {
                const size_t lstride = (size_t)Hkv * kv->cap * D;   // one slot
                HIP_TRY(launch_kv_rope_append(st->pf_qkv, nqkv, (const int*)(db + off_pos) + p0, st->rope, pr, P0 + p0, Hq, Hkv,
                                              D, kv->kc + (size_t)l * lstride, kv->vc + (size_t)l * lstride, kv->cap,
                                              first ? kv->table[kv->cur] : nullptr, dt_code(c.kv_dtype), s));
                const int q0 = p0 / PF_ATT_ROWS, nq = (pr + PF_ATT_ROWS - 1) / PF_ATT_ROWS;
                AttnArgs a{};
                a.qkv = st->pf_qkv;
                a.qkv_ld = nqkv;
                a.out = st->pf_act;                                  // scratch: the gate|up product rewrites it
                a.out_ld = Hq * D;
                a.meta.reqs = (const ReqDev*)(db + off_req) + q0;
                a.meta.items = (const ItemDev*)(db + off_item) + q0;
                a.meta.positions = (const int*)(db + off_pos) + p0;
                a.meta.row_item = (const int*)(db + off_ritem) + p0;
                a.meta.masks = db + off_mask;
                a.meta.n_items = nq;
                a.meta.M = pr;
                a.meta.n_req = nq;
                a.rope = st->rope;
                a.layer = l;
                a.Hq = Hq;
                a.Hkv = Hkv;
                a.kv_dt = dt_code(c.kv_dtype);
                a.qscale = (float)(1.4426950408889634 / std::sqrt((double)D));
                a.part = st->apart;
                a.counters = st->acnt;
                a.nsplit_max = splits;
                a.vector_path = st->attn_vector;
                {                                            // the direct-load form: the longest chunk's split fits
                    const int Lmax = P0 + p0 + pr;
                    int sl = std::max(ATTN_MIN_SPLIT, (Lmax + splits - 1) / splits);
                    sl = (sl + KGROUPS - 1) / KGROUPS * KGROUPS;
                    a.dma = st->attn_dma && sl <= 1024 && lstride * 2 <= 0xFFFFFFF0ull ? 1 : 0;
                }
                a.bp_out = st->pf_bp;
                a.bc_out = st->pf_bc;
                a.kp = kp;
                a.no_append = 1;
                HIP_TRY(launch_attention(a, D, (Hq / Hkv) * PF_ATT_ROWS, s));
            }
            HIP_TRY(prof_mark(st, STAGE_KERNEL_ATTN, false, s));
            // x = residual + o W_o^T
            HIP_TRY(prof_mark(st, STAGE_KERNEL_OPROJ, true, s));
            {
                PfArgs a = pf(Ld.o, pr, EPI_RESID);
                a.out = st->pf_x;
                a.out_ld = H;
                a.resid = first ? (const void*)hin : (const void*)st->pf_x;
                a.resid_dt = first ? act_dt : DT_F32;
                a.resid_ld = H;
                HIP_TRY(launch_gemm_pf(a, s));
            }
            HIP_TRY(prof_mark(st, STAGE_KERNEL_OPROJ, false, s));
            // act = silu(h2 W_g^T) * (h2 W_u^T), h2 = RMSNorm(x)
            HIP_TRY(prof_mark(st, STAGE_KERNEL_GATEUP, true, s));
            HIP_TRY(launch_bprep_rows(st->pf_x, DT_F32, H, Ld.ffn_norm, act_dt, H, c.rms_eps, pr, st->pf_bp, st->pf_bc, kp, s));
            {
                PfArgs a = pf(Ld.gu, pr, EPI_SWIGLU);
                a.out = st->pf_act;
                a.out_ld = F;
                a.n_valid = F;
                HIP_TRY(launch_gemm_pf(a, s));
            }
            HIP_TRY(prof_mark(st, STAGE_KERNEL_GATEUP, false, s));
            // x = x + act W_d^T; the last layer also writes hidden_out
            HIP_TRY(prof_mark(st, STAGE_KERNEL_DOWN, true, s));
            HIP_TRY(launch_bprep_rows(st->pf_act, DT_F32, F, nullptr, act_dt, F, c.rms_eps, pr, st->pf_bp, st->pf_bc, kp, s));
            {
                PfArgs a = pf(Ld.d, pr, EPI_RESID);
                a.out = st->pf_x;
                a.out_ld = H;
                a.resid = st->pf_x;
                a.resid_dt = DT_F32;
                a.resid_ld = H;
                if (last) {
                    a.out_act = (uint8_t*)hidden_out + (size_t)p0 * row_bytes;
                    a.out_act_dt = act_dt;
                    a.out_act_ld = H;
                }
                HIP_TRY(launch_gemm_pf(a, s));
            }
            HIP_TRY(prof_mark(st, STAGE_KERNEL_DOWN, false, s));
        }
    }
    HIP_TRY(mark_done(st, s));
    kv->P = P0 + n;
    return STAGE_OK;
}

int stage_debug_dequant(Stage* stage, int layer, int which, float* out_host) {
    if (!stage || !out_host) return fail(STAGE_E_INVALID, "NULL argument");
    const StageConfig& c = stage->cfg;
    const bool row_layout = which >= 8;
    if (row_layout) which -= 8;
    if (layer < 0 || layer >= c.n_layers || which < 0 || which > 6) return fail(STAGE_E_INVALID, "layer or matrix index out of range");
    if (row_layout && !stage->ps_ok) return fail(STAGE_E_UNSUPPORTED, "this stage keeps no row-layout weights");
    HIP_TRY(hipSetDevice(stage->device));
    const LayerDev& L = stage->layers[layer];
    const int QD = c.n_q_heads * c.head_dim, KVD = c.n_kv_heads * c.head_dim;
    if (row_layout) {
        const PsLayer& P = stage->ps_host[layer];
        const PsMat* pm = nullptr;
        int off = 0, map = 0, nr = 0, kc = stage->kc_h, ng = stage->ng_h, k = c.hidden;
        switch (which) {
            case 0: pm = &P.qkv; map = 3; nr = QD; break;
            case 1: pm = &P.qkv; map = 3; off = QD; nr = KVD; break;
            case 2: pm = &P.qkv; map = 3; off = QD + KVD; nr = KVD; break;
            case 3: pm = &P.o; nr = c.hidden; kc = stage->kc_q; ng = stage->ng_q; k = QD; break;
            case 4: pm = &P.gu; map = 1; nr = c.ffn; break;
            case 5: pm = &P.gu; map = 2; nr = c.ffn; break;
            default: pm = &P.d; nr = c.hidden; kc = stage->kc_f; ng = stage->ng_f; k = c.ffn; break;
        }
        float* tmp = nullptr;
        const size_t bytes = (size_t)nr * k * sizeof(float);
        if (hipMalloc(&tmp, bytes) != hipSuccess) {
            (void)hipGetLastError();
            return fail(STAGE_E_OOM, "staging allocation failed");
        }
        hipError_t e = launch_dequant_rows(*pm, kc, ng, c.group_size / CHUNK_K, k, off, map, nr, c.head_dim, tmp, nullptr);
        if (e == hipSuccess) e = hipMemcpy(out_host, tmp, bytes, hipMemcpyDeviceToHost);
        (void)hipFree(tmp);
        if (e != hipSuccess) return fail(STAGE_E_HIP, std::string("debug dequant: ") + hipGetErrorString(e));
        return STAGE_OK;
    }
    const PackedMat* m = nullptr;
    int off = 0, map = 0, rows = 0;
    switch (which) {
        case 0: m = &L.qkv.pm; off = 0; rows = QD; break;
        case 1: m = &L.qkv.pm; off = QD; rows = KVD; break;
        case 2: m = &L.qkv.pm; off = QD + KVD; rows = KVD; break;
        case 3: m = &L.o.pm; rows = c.hidden; break;
        case 4: m = &L.gu.pm; map = 1; rows = c.ffn; break;
        case 5: m = &L.gu.pm; map = 2; rows = c.ffn; break;
        default: m = &L.d.pm; rows = c.hidden; break;
    }
    float* tmp = nullptr;
    const size_t bytes = (size_t)rows * m->k * sizeof(float);
    if (hipMalloc(&tmp, bytes) != hipSuccess) {
        (void)hipGetLastError();
        return fail(STAGE_E_OOM, "staging allocation failed");
    }
    hipError_t e = launch_dequant(*m, off, map, rows, tmp, nullptr);
    if (e == hipSuccess) e = hipMemcpy(out_host, tmp, bytes, hipMemcpyDeviceToHost);
    (void)hipFree(tmp);
    if (e != hipSuccess) return fail(STAGE_E_HIP, std::string("debug dequant: ") + hipGetErrorString(e));
    return STAGE_OK;
}

int stage_forward(Stage* st, const StageRequest* reqs, int n_req, const void* hidden_in, void* hidden_out, void* stream) {
    if (!st || !reqs || !hidden_in || !hidden_out) return fail(STAGE_E_INVALID, "NULL argument");
    if (n_req < 1) return fail(STAGE_E_INVALID, "n_req must be positive");
    const StageConfig& c = st->cfg;
    const int H = c.hidden, D = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads, F = c.ffn;
    const int gs = Hq / Hkv;

    // ---------------- validation (no side effects)
    int M = 0, n_items = 0, max_queries_item = 0, max_splits = 1;
    size_t mask_bytes = 0, beam_ints = 0;
    for (int r = 0; r < n_req; ++r) {
        const StageRequest& q = reqs[r];
        const std::string who = "request " + std::to_string(r) + ": ";
        if (!q.state) return fail(STAGE_E_INVALID, who + "state is NULL");
        if (q.state->stage != st) return fail(STAGE_E_STATE_MISMATCH, who + "state belongs to another stage");
        for (int r2 = 0; r2 < r; ++r2)
            if (reqs[r2].state == q.state) return fail(STAGE_E_STATE_MISMATCH, who + "state used twice in one forward");
        const int S = q.state->S, n = q.n_tokens, P = q.state->P;
        if (n < 1) return fail(STAGE_E_INVALID, who + "n_tokens must be positive");
        if (!q.positions || (!q.attention_mask && !q.attention_mask_rows))
            return fail(STAGE_E_INVALID, who + "positions and a mask (attention_mask or attention_mask_rows) are required");
        if (q.mask_len != P + n)
            return fail(STAGE_E_SHAPE, who + "mask_len " + std::to_string(q.mask_len) + " != P + n = " + std::to_string(P + n));
        if (P + n > q.state->cap) return fail(STAGE_E_CAPACITY, who + "P + n exceeds the state's capacity");
        for (int i = 0; i < S * n; ++i)
            if (q.positions[i] < 0 || q.positions[i] >= c.max_positions)
                return fail(STAGE_E_CAPACITY, who + "position " + std::to_string(q.positions[i]) + " outside the rotary table");
        if (q.beam_idx)
            for (int b = 0; b < S; ++b)
                if (q.beam_idx[b] < 0 || q.beam_idx[b] >= S) return fail(STAGE_E_INVALID, who + "beam_idx out of range");
        for (int b = 0; b < S; ++b) {
            const uint8_t* mk = q.attention_mask ? q.attention_mask + (size_t)b * q.mask_len : nullptr;
            if (!q.attention_mask_rows) {
                int first = -1;
                for (int j = 0; j < P + n; ++j)
                    if (mk[j]) { first = j; break; }
                if (first < 0 || first > P)   // query 0 sees rows 0..P; later queries see more
                    return fail(STAGE_E_INVALID, who + "slot " + std::to_string(b) + " has a query row with no visible key");
                continue;
            }
            for (int i = 0; i < n; ++i) {     // each query row: some key j <= P + i kept by both masks
                const uint8_t* rw = q.attention_mask_rows + ((size_t)b * n + i) * q.mask_len;
                bool any = false;
                for (int j = 0; j <= P + i && !any; ++j) any = rw[j] && (!mk || mk[j]);
                if (!any)
                    return fail(STAGE_E_INVALID, who + "slot " + std::to_string(b) + " query " + std::to_string(i) +
                                                     " sees no key");
            }
        }
        M += S * n;
        n_items += S;
        max_queries_item = std::max(max_queries_item, gs * n);
        mask_bytes += (size_t)S * q.mask_len * (q.attention_mask_rows ? (size_t)(1 + n) : 1);
        if (q.beam_idx) beam_ints += S;
    }
    if (M > MAX_ROWS) return fail(STAGE_E_CAPACITY, "total rows " + std::to_string(M) + " exceed STAGE_MAX_ROWS");
    if ((const uint8_t*)hidden_in < (const uint8_t*)hidden_out + (size_t)M * H * 2 &&
        (const uint8_t*)hidden_out < (const uint8_t*)hidden_in + (size_t)M * H * 2)
        return fail(STAGE_E_INVALID, "hidden_in and hidden_out overlap");

    HIP_TRY(hipSetDevice(st->device));
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(order_on(st, s));

    // ---------------- metadata into a pinned ring slot, one H2D copy
    const size_t off_req = 0;
    const size_t off_item = align16(off_req + sizeof(ReqDev) * n_req);
    const size_t off_pos = align16(off_item + sizeof(ItemDev) * n_items);
    const size_t off_ritem = align16(off_pos + sizeof(int) * M);
    const size_t off_beam = align16(off_ritem + sizeof(int) * M);
    const size_t off_mask = align16(off_beam + sizeof(int) * beam_ints);
    const size_t total = align16(off_mask + mask_bytes);
    int rc = ensure_meta(st, total);
    if (rc) return rc;
    const int slot_i = st->ring_i;
    st->ring_i = (st->ring_i + 1) % META_RING;
    if (st->meta_ev_used[slot_i]) HIP_TRY(hipEventSynchronize(st->meta_ev[slot_i]));
    uint8_t* hb = st->meta_host[slot_i];
    ReqDev* rd = (ReqDev*)(hb + off_req);
    ItemDev* id = (ItemDev*)(hb + off_item);
    int* pos = (int*)(hb + off_pos);
    int* ritem = (int*)(hb + off_ritem);
    int* beam = (int*)(hb + off_beam);
    uint8_t* masks = hb + off_mask;
    std::vector<int> beam_off(n_req, -1);
    std::vector<bool> do_gather(n_req, false);
    bool attn_dma_ok = st->attn_dma;
    {
        int row = 0, item = 0;
        size_t moff = 0, boff = 0;
        for (int r = 0; r < n_req; ++r) {
            const StageRequest& q = reqs[r];
            KVState* kv = q.state;
            const int S = kv->S, n = q.n_tokens;
            bool ident = true;
            if (q.beam_idx)
                for (int b = 0; b < S; ++b) ident = ident && (q.beam_idx[b] == b);
            do_gather[r] = !ident && kv->P > 0;
            if (q.beam_idx) {
                beam_off[r] = (int)boff;
                std::memcpy(beam + boff, q.beam_idx, sizeof(int) * S);
                boff += S;
            }
            ReqDev& d = rd[r];
            d.P = kv->P;
            d.n = n;
            d.S = S;
            d.row0 = row;
            d.cap = kv->cap;
            d.mask_off = (int)moff;
            d.mask_len = q.mask_len;
            d.rowmask_off = q.attention_mask_rows ? (int)(moff + (size_t)S * q.mask_len) : -1;   // rows follow the slot masks
            d.item0 = item;
            // attention splits: about two workgroups per CU over the request's own
            // slots and kv heads (never its batch-mates, so they cannot change its
            // result), at most ATTN_MAX_SPLITS
            d.splits = std::max(1, std::min(ATTN_MAX_SPLITS, 2 * st->n_cus / (S * Hkv)));
            if (const char* e = std::getenv("STAGE_ATTN_SPLITS")) d.splits = std::max(1, std::min(ATTN_MAX_SPLITS, atoi(e)));
            max_splits = std::max(max_splits, d.splits);
            {                                            // the direct-load attention stages a whole split's table
                const int Lr = d.P + n;
                int sl = std::max(ATTN_MIN_SPLIT, (Lr + d.splits - 1) / d.splits);
                sl = (sl + KGROUPS - 1) / KGROUPS * KGROUPS;
                // and addresses one layer of the cache through a buffer resource (32-bit offsets)
                const size_t layer_bytes = (size_t)S * Hkv * kv->cap * c.head_dim * 2;
                // and the split's rows of a per-query-row mask (n rows x split keys, at most 8 KB)
                const bool rows_fit = !q.attention_mask_rows || (size_t)n * ((sl + 3) / 4 * 4) <= 8192;
                if (sl > 1024 || !rows_fit || layer_bytes > 0xFFFFFFF0ull) attn_dma_ok = false;
            }
            d.kc = kv->kc;
            d.vc = kv->vc;
            d.table = kv->table[do_gather[r] ? 1 - kv->cur : kv->cur];
            for (int b = 0; b < S; ++b) {
                id[item + b] = ItemDev{r, b, d};
                for (int i = 0; i < n; ++i) ritem[row + b * n + i] = item + b;
            }
            std::memcpy(pos + row, q.positions, sizeof(int) * S * n);
            if (!q.attention_mask_rows) {
                std::memcpy(masks + moff, q.attention_mask, (size_t)S * q.mask_len);
            } else {
                // slot mask: the keys some row of the slot keeps (and the 2-D mask keeps);
                // the rows follow, each refined by the 2-D mask
                const size_t ml = (size_t)q.mask_len;
                uint8_t* sm = masks + moff;
                uint8_t* rm = sm + (size_t)S * ml;
                for (int b = 0; b < S; ++b)
                    for (size_t j = 0; j < ml; ++j) {
                        const bool keep2 = !q.attention_mask || q.attention_mask[b * ml + j];
                        uint8_t any = 0;
                        for (int i = 0; i < n; ++i) {
                            const uint8_t v = (keep2 && q.attention_mask_rows[((size_t)b * n + i) * ml + j]) ? 1 : 0;
                            rm[((size_t)b * n + i) * ml + j] = v;
                            any |= v;
                        }
                        sm[b * ml + j] = any;
                    }
                moff += (size_t)S * n * ml;
            }
            row += S * n;
            item += S;
            moff += (size_t)S * q.mask_len;
        }
    }
    uint8_t* db = st->meta_dev;
    HIP_TRY(hipMemcpyAsync(db, hb, total, hipMemcpyHostToDevice, s));
    HIP_TRY(hipEventRecord(st->meta_ev[slot_i], s));
    st->meta_ev_used[slot_i] = true;

    // ---------------- beam reorder of the index tables (rows are never copied)
    for (int r = 0; r < n_req; ++r) {
        if (!do_gather[r]) continue;
        KVState* kv = reqs[r].state;
        HIP_TRY(launch_table_gather(kv->table[kv->cur], kv->table[1 - kv->cur], (const int*)(db + off_beam) + beam_off[r],
                                    kv->S, kv->cap, kv->P, s));
    }

    MetaDev meta;
    meta.reqs = (const ReqDev*)(db + off_req);
    meta.items = (const ItemDev*)(db + off_item);
    meta.positions = (const int*)(db + off_pos);
    meta.row_item = (const int*)(db + off_ritem);
    meta.masks = db + off_mask;
    meta.n_items = n_items;
    meta.M = M;
    meta.n_req = n_req;

    const int act_dt = dt_code(c.act_dtype);
    const int nqkv = Hq * D + 2 * Hkv * D;

    // ---------------- one launch for the whole stage: a single decode row
    const int RPS = 512 / D;                               // cache rows per 1 KB slot
    int nsplit = 0, split_len = 0, att_T = 0;
    bool single = st->ps_ok && M == 1 && (st->prof_class < 0 || st->prof_class == STAGE_KERNEL_PERSISTENT);
    if (single) {
        const int P = reqs[0].state->P;
        // splits per kv head: a power of two; each split's merge slice is a multiple of 8 outputs
        const int max_split = std::min(st->ps_nwg / Hkv, gs * D / 8);
        int cap_split = 32;
        if (const char* e = std::getenv("STAGE_ATTN_SPLITS")) cap_split = std::max(1, atoi(e));
        nsplit = 1;
        while (nsplit * 2 <= std::min(cap_split, max_split)) nsplit *= 2;
        for (;;) {
            split_len = (P + nsplit - 1) / nsplit;
            att_T = ((split_len + SK_CW - 1) / SK_CW + RPS - 1) / RPS;
            if (att_T <= SK_TMAX || nsplit * 2 > max_split) break;
            nsplit *= 2;
        }
        if (att_T > SK_TMAX) single = false;               // cache too long for one pass: per-layer kernels
    }
    if (single) {
        PsArgs a{};
        a.layers = st->ps_layers;
        for (int m = 0; m < 4; ++m) {
            a.wb[m] = st->ps_wb[m];
            a.wl[m] = st->ps_wl[m];
        }
        a.n_layers = c.n_layers;
        a.H = H; a.Hq = Hq; a.Hkv = Hkv; a.F = F; a.QD = Hq * D; a.NQKV = nqkv;
        a.kc_h = st->kc_h; a.kc_q = st->kc_q; a.kc_f = st->kc_f;
        a.ng_h = st->ng_h; a.ng_q = st->ng_q; a.ng_f = st->ng_f;
        a.gchunks = c.group_size / CHUNK_K;
        a.eps = c.rms_eps;
        a.act_dt = act_dt;
        a.kv_dt = dt_code(c.kv_dtype);
        a.hidden_in = hidden_in;
        a.hidden_out = hidden_out;
        a.rpw_qkv = st->ps_rpw_qkv; a.rpw_h = st->ps_rpw_h; a.rpw_gu = st->ps_rpw_gu;
        a.ll_x = st->ll_x; a.ll_qkv = st->ll_qkv; a.ll_o = st->ll_o; a.ll_act = st->ll_act;
        a.meta = meta;
        a.rope = st->rope;
        a.qscale = (float)(1.4426950408889634 / std::sqrt((double)D));
        a.nsplit = nsplit; a.split_len = split_len; a.att_T = att_T;
        a.ll_part = st->ll_part;
        a.ll_epoch = st->ll_epoch;
        a.err = st->err;
        a.spin_limit = st->spin_limit;
        a.trace = st->trace;
        a.dbg_layer = -1;
        if (st->dbg_layer >= 0) {                         // test support: record one layer's queries and scores
            HIP_TRY(launch_fill_u32((uint32_t*)st->dbg_logits, (size_t)Hq * st->dbg_keys, 0xFFFFFFFFu, s));   // NaN
            a.dbg_q = st->dbg_q;
            a.dbg_logits = st->dbg_logits;
            a.dbg_keys = st->dbg_keys;
            a.dbg_layer = st->dbg_layer;
            st->dbg_rows = 1;
        }
        const int kvb = c.kv_dtype == STAGE_DTYPE_BF16;
        const int lds = ps_layout(a, ps_slots(st->cpl_h, st->cpl_q, st->cpl_f, D, gs, kvb), D, gs);
        HIP_TRY(prof_mark(st, STAGE_KERNEL_PERSISTENT, true, s));
        hipError_t e = launch_persistent(a, st->cpl_h, st->cpl_q, st->cpl_f, D, gs, kvb, st->ps_nwg, (size_t)lds, st->ps_coop, s);
        if (e != hipSuccess) return fail(STAGE_E_HIP, std::string("single-launch forward: ") + hipGetErrorString(e));
        HIP_TRY(prof_mark(st, STAGE_KERNEL_PERSISTENT, false, s));
        st->ll_epoch += (unsigned)(PS_LL_PER_LAYER * c.n_layers);
        HIP_TRY(mark_done(st, s));
        for (int r = 0; r < n_req; ++r) {
            KVState* kv = reqs[r].state;
            if (do_gather[r]) kv->cur = 1 - kv->cur;
            kv->P += reqs[r].n_tokens;
        }
        return STAGE_OK;
    }
    auto run_gemv = [&](const DevMat& m, GemvArgs a, size_t in_row_elems, size_t out_row_elems, size_t resid_row_elems,
                        int in_elem_bytes, int resid_elem_bytes) -> hipError_t {
        a.W = m.pm;
        a.ksplit = m.ksplit;
        a.cps = m.cps;
        a.partial = st->gpart;
        a.counters = st->gcnt;
        for (int m0 = 0; m0 < M; m0 += GEMV_MAX_M) {
            GemvArgs b = a;
            b.M = std::min(GEMV_MAX_M, M - m0);
            b.in = (const uint8_t*)a.in + (size_t)m0 * in_row_elems * in_elem_bytes;
            b.out = a.out + (size_t)m0 * out_row_elems;
            if (a.resid) b.resid = (const uint8_t*)a.resid + (size_t)m0 * resid_row_elems * resid_elem_bytes;
            if (a.ssq_in) b.ssq_in = a.ssq_in + (size_t)m0 * a.ssq_tiles;
            if (a.ssq_out) b.ssq_out = a.ssq_out + (size_t)m0 * m.pm.ntiles;
            if (a.out_act) b.out_act = (uint8_t*)a.out_act + (size_t)m0 * a.out_act_ld * 2;
            hipError_t e = launch_gemv(b, s);
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    };

    // 2..64 rows: each product reads its input prepared by the kernel before it
    const bool use_bp = st->bp_ok && M >= st->gemm_min_rows && M <= MAX_ROWS;
    int bcur = 0;                                           // buffer holding the next product's input
    auto bp_in = [&](GemvArgs& a, int norm) {
        a.bp_in = st->bp[bcur];
        a.bc_in = st->bc[bcur];
        a.cb_in = st->cbf[bcur];
        a.norm = norm;
    };
    auto bp_out = [&](GemvArgs& a) {
        a.bp_out = st->bp[1 - bcur];
        a.bc_out = st->bc[1 - bcur];
        a.cb_out = st->cbf[1 - bcur];
    };
    auto run_bp = [&](const DevMat& m, GemvArgs a) -> hipError_t {
        a.W = m.pm;
        a.M = M;
        a.kp = st->kp;
        a.partial = st->gpart;
        a.counters = st->gcnt;
        a.ksplit = m.bp_split;
        a.kg = m.bp_kg;
        return launch_gemm_bp(a, s);
    };

    for (int l = 0; l < c.n_layers; ++l) {
        const LayerDev& Ld = st->layers[l];
        const bool first = (l == 0), last = (l == c.n_layers - 1);
        // q|k|v = RMSNorm(x) W_qkv^T
        if (use_bp) {
            GemvArgs a{};
            a.eps = c.rms_eps;
            a.ssq_in = st->ssq;
            a.ssq_tiles = st->ntiles_h;
            a.epi = EPI_STORE;
            a.out = st->qkv;
            a.out_ld = nqkv;
            HIP_TRY(prof_mark(st, STAGE_KERNEL_QKV, true, s));
            if (first) {
                HIP_TRY(launch_bprep(hidden_in, act_dt, H, Ld.attn_norm, act_dt, H, c.rms_eps, M, st->bp[bcur], st->bc[bcur],
                                     st->kp, st->rsb, s));
                bp_in(a, 2);
            } else {
                bp_in(a, 1);
                a.rs_out = st->rsb;
            }
            HIP_TRY(run_bp(Ld.qkv, a));
            HIP_TRY(prof_mark(st, STAGE_KERNEL_QKV, false, s));
        } else {
            GemvArgs a{};
            a.in = first ? hidden_in : (const void*)st->x;
            a.in_dt = first ? act_dt : DT_F32;
            a.in_ld = H;
            a.gamma = Ld.attn_norm;
            a.gamma_dt = act_dt;
            a.rms = first ? RMS_FULLROW : RMS_PARTIALS;
            a.eps = c.rms_eps;
            a.ssq_in = first ? nullptr : st->ssq;
            a.ssq_tiles = st->ntiles_h;
            a.epi = EPI_STORE;
            a.out = st->qkv;
            a.out_ld = nqkv;
            HIP_TRY(prof_mark(st, STAGE_KERNEL_QKV, true, s));
            HIP_TRY(run_gemv(Ld.qkv, a, H, nqkv, 0, first ? 2 : 4, 0));
            HIP_TRY(prof_mark(st, STAGE_KERNEL_QKV, false, s));
        }
        // attention (rotary, append, mask, online softmax, split merge)
        {
            AttnArgs a{};
            a.qkv = st->qkv;
            a.qkv_ld = nqkv;
            a.out = st->attn;
            a.out_ld = Hq * D;
            a.meta = meta;
            a.rope = st->rope;
            a.layer = l;
            a.Hq = Hq;
            a.Hkv = Hkv;
            a.kv_dt = dt_code(c.kv_dtype);
            a.qscale = (float)(1.4426950408889634 / std::sqrt((double)D));
            a.part = st->apart;
            a.counters = st->acnt;
            // splits per (slot, kv head) follow the request's own length and slot count
            // only (at least ATTN_MIN_SPLIT keys each, at most its `splits`), so
            // batch-mates never change a request's result; nsplit_max bounds the grid
            // and is the stride of the partials
            a.nsplit_max = max_splits;
            a.vector_path = st->attn_vector;
            a.dma = attn_dma_ok ? 1 : 0;
            if (l == st->dbg_layer && !st->attn_vector) {    // test support: record this layer's queries and scores
                HIP_TRY(launch_fill_u32((uint32_t*)st->dbg_logits, (size_t)M * Hq * st->dbg_keys, 0xFFFFFFFFu, s));   // NaN
                a.dbg_q = st->dbg_q;
                a.dbg_logits = st->dbg_logits;
                a.dbg_keys = st->dbg_keys;
                st->dbg_rows = M;
            }
            if (use_bp) {
                a.bp_out = st->bp[1 - bcur];
                a.bc_out = st->bc[1 - bcur];
                a.kp = st->kp;
            }
            HIP_TRY(prof_mark(st, STAGE_KERNEL_ATTN, true, s));
            HIP_TRY(launch_attention(a, D, max_queries_item, s));
            HIP_TRY(prof_mark(st, STAGE_KERNEL_ATTN, false, s));
            if (use_bp) bcur = 1 - bcur;
        }
        // x = residual + o W_o^T
        {
            GemvArgs a{};
            a.in = st->attn;
            a.in_dt = DT_F32;
            a.in_ld = Hq * D;
            a.rms = RMS_NONE;
            a.epi = EPI_RESID;
            a.out = st->x;
            a.out_ld = H;
            a.resid = first ? hidden_in : (const void*)st->x;
            a.resid_dt = first ? act_dt : DT_F32;
            a.resid_ld = H;
            a.ssq_out = st->ssq;
            HIP_TRY(prof_mark(st, STAGE_KERNEL_OPROJ, true, s));
            if (use_bp) {                                   // also prepares RMSNorm_ffn's input (c = rs_attn)
                bp_in(a, 0);
                bp_out(a);
                a.gamma_next = Ld.ffn_norm;
                a.gamma_next_dt = act_dt;
                a.rs_in = st->rsb;
                HIP_TRY(run_bp(Ld.o, a));
                bcur = 1 - bcur;
            } else {
                HIP_TRY(run_gemv(Ld.o, a, Hq * D, H, H, 4, first ? 2 : 4));
            }
            HIP_TRY(prof_mark(st, STAGE_KERNEL_OPROJ, false, s));
        }
        // act = silu(h2 W_g^T) * (h2 W_u^T), h2 = RMSNorm(x)
        {
            GemvArgs a{};
            a.in = st->x;
            a.in_dt = DT_F32;
            a.in_ld = H;
            a.gamma = Ld.ffn_norm;
            a.gamma_dt = act_dt;
            a.rms = RMS_PARTIALS;
            a.eps = c.rms_eps;
            a.ssq_in = st->ssq;
            a.ssq_tiles = st->ntiles_h;
            a.epi = EPI_SWIGLU;
            a.out = st->act;
            a.out_ld = F;
            a.n_valid = F;
            HIP_TRY(prof_mark(st, STAGE_KERNEL_GATEUP, true, s));
            if (use_bp) {                                   // also prepares the down product's input
                bp_in(a, 1);
                bp_out(a);
                a.rs_out = st->rsb;
                HIP_TRY(run_bp(Ld.gu, a));
                bcur = 1 - bcur;
            } else {
                HIP_TRY(run_gemv(Ld.gu, a, H, F, 0, 4, 0));
            }
            HIP_TRY(prof_mark(st, STAGE_KERNEL_GATEUP, false, s));
        }
        // x = x + act W_d^T  (last layer also writes hidden_out)
        {
            GemvArgs a{};
            a.in = st->act;
            a.in_dt = DT_F32;
            a.in_ld = F;
            a.rms = RMS_NONE;
            a.epi = EPI_RESID;
            a.out = st->x;
            a.out_ld = H;
            a.resid = st->x;
            a.resid_dt = DT_F32;
            a.resid_ld = H;
            a.ssq_out = st->ssq;
            if (last) {
                a.out_act = hidden_out;
                a.out_act_dt = act_dt;
                a.out_act_ld = H;
            }
            HIP_TRY(prof_mark(st, STAGE_KERNEL_DOWN, true, s));
            if (use_bp) {                                   // also prepares the next layer's q|k|v input (c = rs_ffn)
                bp_in(a, 0);
                if (!last) {
                    bp_out(a);
                    a.gamma_next = st->layers[l + 1].attn_norm;
                    a.gamma_next_dt = act_dt;
                    a.rs_in = st->rsb;
                }
                HIP_TRY(run_bp(Ld.d, a));
                if (!last) bcur = 1 - bcur;
            } else {
                HIP_TRY(run_gemv(Ld.d, a, F, H, H, 4, 4));
            }
            HIP_TRY(prof_mark(st, STAGE_KERNEL_DOWN, false, s));
        }
    }

    // ---------------- commit host-side state
    HIP_TRY(mark_done(st, s));
    for (int r = 0; r < n_req; ++r) {
        KVState* kv = reqs[r].state;
        if (do_gather[r]) kv->cur = 1 - kv->cur;
        kv->P += reqs[r].n_tokens;
    }
    return STAGE_OK;
}

}  // extern "C"
