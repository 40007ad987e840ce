// C ABI of the three-stage W4A16 decoder layer (declared in include/w4layer.h):
// argument validation, weight repacking into the tiled device layout, the
// workspace plan and the kernel sequence of each stage.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdarg>
#include <cstring>
#include <mutex>
#include <string>
#include <thread>
#include <vector>
#include <unistd.h>

#include "../../include/w4layer.h"
#include "common.h"
#include "decode_fused.h"
#include "launch.h"
#include "lm.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

#define HIP_TRY(call)                                                                        \
    do {                                                                                     \
        hipError_t e_ = (call);                                                              \
        if (e_ != hipSuccess) return fail(W4_EHIP, "%s: %s", #call, hipGetErrorString(e_)); \
    } while (0)

int round_up(int a, int b) { return (a + b - 1) / b * b; }

struct DevBuf {
    void* p = nullptr;
    ~DevBuf() { if (p) (void)hipFree(p); }
};

// Canonical host linear (see qlinear_host) with its logical shape.
struct HostLin {
    const int32_t* qw;
    const uint16_t* sc;
    const uint8_t* z;
    int K, N;
    int fmt = W4_WEIGHTS_INT4;
    const uint8_t* q8 = nullptr;
    const uint16_t* w16 = nullptr;
};

struct ColSrc {        // where a device column comes from
    const HostLin* lin;  // null: padding column
    int n;
};

struct Repacked {
    std::vector<uint32_t> qw;
    std::vector<uint16_t> scales;
    std::vector<float> ratios;
    std::vector<uint8_t> zeros;
    std::vector<uint32_t> sz;
};

inline bool f16_is_zero(uint16_t b) { return (b & 0x7FFFu) == 0; }
inline double f16_value(uint16_t b) {
    const int e = (b >> 10) & 0x1F, f = b & 0x3FF;
    const double v = (e == 0) ? std::ldexp((double)f, -24) : std::ldexp(1.0 + f / 1024.0, e - 15);
    return (b & 0x8000u) ? -v : v;
}

// Repack columns [c0, c1) of a device linear with N_dev columns.
void repack_cols(const std::vector<ColSrc>& cols, int K_pad, int G, bool has_zeros, Repacked& R, int c0, int c1) {
    const int KG = K_pad / G, KB = K_pad / 64;
    const size_t N_dev = cols.size();
    std::vector<uint8_t> code(K_pad);
    std::vector<uint16_t> s(KG);
    std::vector<uint8_t> z(KG);
    std::vector<char> dead(KG);
    for (int nd = c0; nd < c1; nd++) {
        const ColSrc& cs = cols[nd];
        const HostLin* L = cs.lin;
        const int ng = L ? (L->K + G - 1) / G : 0;
        for (int g = 0; g < KG; g++) {
            s[g] = (L && g < ng) ? L->sc[(size_t)g * L->N + cs.n] : 0;
            z[g] = (L && L->z && g < ng) ? L->z[(size_t)g * L->N + cs.n] : 8;
            dead[g] = f16_is_zero(s[g]);
        }
        // non-zero stand-in scales for groups that contribute nothing
        uint16_t first = 0x3C00;
        for (int g = 0; g < KG; g++)
            if (!dead[g]) { first = s[g]; break; }
        uint16_t prev = first;
        for (int g = 0; g < KG; g++) {
            if (dead[g]) s[g] = prev; else prev = s[g];
        }
        for (int k = 0; k < K_pad; k++) {
            const int g = k / G;
            uint8_t cv = z[g];
            if (L && k < L->K && !dead[g]) {
                const uint32_t w = (uint32_t)L->qw[(size_t)(k / 8) * L->N + cs.n];
                cv = (w >> (4 * (k % 8))) & 0xF;
            }
            code[k] = cv;
        }
        const int nb = nd / 32, cc = nd % 32;
        for (int kb = 0; kb < KB; kb++)
            for (int hh = 0; hh < 2; hh++)
                for (int si = 0; si < 4; si++) {
                    const int k0 = kb * 64 + si * 16 + hh * 8;
                    uint32_t w = 0;
                    for (int j = 0; j < 8; j++) w |= (uint32_t)code[k0 + j] << (4 * (j / 2) + 16 * (j % 2));
                    R.qw[(((size_t)nb * KB + kb) * 64 + hh * 32 + cc) * 4 + si] = w;
                }
        for (int g = 0; g < KG; g++) {
            const size_t gi = (size_t)g * N_dev + nd;
            R.scales[gi] = s[g];
            R.ratios[gi] = g == 0 ? 1.0f : (float)(f16_value(s[g - 1]) / f16_value(s[g]));
            if (has_zeros) {
                R.zeros[gi] = z[g];
                R.sz[gi] = (uint32_t)s[g] | ((uint32_t)z[g] << 16);
            }
        }
    }
}

// fp16 bits of a double (round to nearest even, subnormals; the caller keeps
// |v| within the finite range).
uint16_t f16_bits(double v) {
    uint16_t sign = std::signbit(v) ? 0x8000u : 0u;
    double a = std::fabs(v);
    if (a == 0.0) return sign;
    int e;
    std::frexp(a, &e);                     // a = m 2^e, 0.5 <= m < 1
    const int ex = std::max(e - 1, -14);   // fp16 exponent (subnormals at -14)
    const double q = std::nearbyint(std::ldexp(a, 10 - ex));   // significand on the 2^(ex-10) grid
    const double r = std::ldexp(q, ex - 10);
    if (r == 0.0) return sign;             // below half the smallest subnormal
    if (r >= 65536.0) return sign | 0x7C00u;
    // encode r exactly
    int e2;
    std::frexp(r, &e2);
    const int ex2 = e2 - 1;
    if (ex2 < -14) return sign | (uint16_t)std::ldexp(r, 24);                       // subnormal
    const uint16_t mant = (uint16_t)(std::ldexp(r, 10 - ex2) - 1024.0);
    return sign | (uint16_t)((ex2 + 15) << 10) | mant;
}

inline double bf16_value(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return (double)f;
}

// Repack columns [c0, c1) of an INT8 (wf 1) or F16 (wf 2) device linear
// (tile layouts of WeightFormat): INT8 codes as unsigned bytes (symmetric
// ones + 128) with the column's scale and zero point in every group of 128;
// F16 values from the bf16 weights, those at k % 8 in {2, 3, 6, 7} times 16.
void repack_cols_x(const std::vector<ColSrc>& cols, int K_pad, int wf, Repacked& R, int c0, int c1) {
    const int KG = K_pad / 128, KB = K_pad / 64;
    const size_t N_dev = cols.size();
    const size_t tile_words = wf == 1 ? 512 : 1024;
    for (int nd = c0; nd < c1; nd++) {
        const ColSrc& cs = cols[nd];
        const HostLin* L = cs.lin;
        uint16_t sc = 0x3C00;
        uint8_t z = 128;
        bool dead = L == nullptr;
        if (wf == 1 && L) {
            sc = L->sc[cs.n];
            if (L->z) z = L->z[cs.n];
            dead = f16_is_zero(sc);
            if (dead) sc = 0x3C00;            // a zero column: codes at the zero point
        }
        const int nb = nd / 32, cc = nd % 32;
        for (int kb = 0; kb < KB; kb++) {
            uint32_t* tile = R.qw.data() + ((size_t)nb * KB + kb) * tile_words;
            for (int hh = 0; hh < 2; hh++)
                for (int si = 0; si < 4; si++) {
                    const int k0 = kb * 64 + si * 16 + hh * 8, lane = hh * 32 + cc;
                    if (wf == 1) {
                        uint32_t wd[2] = {0, 0};
                        for (int j = 0; j < 8; j++) {
                            const int k = k0 + j;
                            uint8_t u = z;
                            if (!dead && k < L->K) {
                                const uint8_t b = L->q8[(size_t)k * L->N + cs.n];
                                u = L->z ? b : (uint8_t)(b ^ 0x80u);
                            }
                            wd[j / 4] |= (uint32_t)u << (8 * (j % 4));
                        }
                        const size_t o = ((size_t)(si / 2) * 64 + lane) * 4 + 2 * (si % 2);
                        tile[o] = wd[0];
                        tile[o + 1] = wd[1];
                    } else {
                        for (int pq = 0; pq < 4; pq++) {
                            uint32_t wd = 0;
                            for (int e = 0; e < 2; e++) {
                                const int k = k0 + 2 * pq + e;
                                double v = 0.0;
                                if (L && k < L->K) v = bf16_value(L->w16[(size_t)k * L->N + cs.n]);
                                if ((pq & 1) == 1) v *= 16.0;
                                wd |= (uint32_t)f16_bits(v) << (16 * e);
                            }
                            tile[((size_t)si * 64 + lane) * 4 + pq] = wd;
                        }
                    }
                }
        }
        for (int g = 0; g < KG; g++) {
            const size_t gi = (size_t)g * N_dev + nd;
            R.scales[gi] = sc;
            R.ratios[gi] = 1.0f;
            if (wf == 1) {
                R.zeros[gi] = z;
                R.sz[gi] = (uint32_t)sc | ((uint32_t)z << 16);
            }
        }
    }
}

}  // namespace

struct DevLinearOwned {
    DevLinear d{};
    DevBuf qw, scales, ratios, zeros, sz, colmap_a, colmap_b, colmap_c;
};

struct Profiler {          // one timed kernel per stage
    static constexpr int kMax = 4096;
    int kernel[3] = {-1, -1, -1};
    int recorded[3] = {-1, -1, -1};  // the kernel whose launches the record holds
    std::vector<hipEvent_t> ev[3];   // 2 per recorded launch
    int used[3] = {0, 0, 0};
    ~Profiler() {
        for (auto& v : ev)
            for (auto e : v) (void)hipEventDestroy(e);
    }
};

// Scratch memory of layer_decode_noalloc: a file-scope device array that each
// device holds from the library's first layer_create on it until the process
// ends.  Host code never passes the array's name to a kernel (on the host it
// names a stand-in, not device memory); it uses the device address that
// hipGetSymbolAddress returned for the current device.
constexpr size_t kScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

constexpr int kMaxBlocks = 1024;                    // persistent decode blocks (one per CU)
constexpr int kSpinDefault = 1 << 20;               // polls per thread per persistent launch
constexpr int kStampWords = 8 + 32 * kMaxBlocks;

struct layer_s {
    layer_config cfg{};
    int F_pad = 0;
    DevLinearOwned qkv, o, gu, down;
    DevBuf attn_norm, mlp_norm, rope_cos, rope_sin;
    int device = 0;
    Profiler prof;
    // persistent decode: error flag and optional per-block time stamps (zeroed)
    DevBuf sync;
    int fused_blocks = 0, S_qkv = 1, S_o = 1, S_down = 1;   // persistent decode: blocks, k parts
    int num_cus = 256;
    int* err = nullptr;
    unsigned long long* stamps = nullptr;
    int decode_path = 0;   // 0 auto, 1 separate kernels, 2 persistent
    bool decode_trace = false;   // persistent decode records its time stamps
    int spin_max = kSpinDefault; // polls per thread per persistent launch before a wait gives up
};

namespace {

int upload(DevBuf& b, const void* src, size_t bytes) {
    if (bytes == 0) return 0;
    HIP_TRY(hipMalloc(&b.p, bytes));
    HIP_TRY(hipMemcpy(b.p, src, bytes, hipMemcpyHostToDevice));
    return 0;
}

int build_linear(DevLinearOwned& out, const std::vector<ColSrc>& cols, int K, int K_pad, int G, bool has_zeros,
                 int fmt = W4_WEIGHTS_INT4) {
    const int N_dev = (int)cols.size();
    const int wf = fmt == W4_WEIGHTS_INT8 ? WF_INT8 : fmt == W4_WEIGHTS_BF16 ? WF_F16 : WF_INT4;
    if (wf != WF_INT4) {
        G = 128;
        has_zeros = wf == WF_INT8;
    }
    const int KG = K_pad / G;
    Repacked R;
    R.qw.resize((size_t)N_dev * K_pad / 8 << wf);
    R.scales.resize((size_t)N_dev * KG);
    R.ratios.resize((size_t)N_dev * KG);
    if (has_zeros) {
        R.zeros.resize((size_t)N_dev * KG);
        R.sz.resize((size_t)N_dev * KG);
    }
    const int nth = std::max(1, std::min(16, (int)std::thread::hardware_concurrency()));
    std::vector<std::thread> th;
    const int per = (N_dev / 32 + nth - 1) / nth * 32;
    for (int i = 0; i < nth; i++) {
        const int c0 = i * per, c1 = std::min(N_dev, (i + 1) * per);
        if (c0 >= c1) break;
        if (wf == WF_INT4) th.emplace_back(repack_cols, std::cref(cols), K_pad, G, has_zeros, std::ref(R), c0, c1);
        else th.emplace_back(repack_cols_x, std::cref(cols), K_pad, wf, std::ref(R), c0, c1);
    }
    for (auto& t : th) t.join();
    int rc;
    if ((rc = upload(out.qw, R.qw.data(), R.qw.size() * 4))) return rc;
    if ((rc = upload(out.scales, R.scales.data(), R.scales.size() * 2))) return rc;
    if ((rc = upload(out.ratios, R.ratios.data(), R.ratios.size() * 4))) return rc;
    if (has_zeros && (rc = upload(out.zeros, R.zeros.data(), R.zeros.size()))) return rc;
    if (has_zeros && (rc = upload(out.sz, R.sz.data(), R.sz.size() * 4))) return rc;
    DevLinear& d = out.d;
    d.qw = (const uint32_t*)out.qw.p;
    d.scales = (const uint16_t*)out.scales.p;
    d.ratios = (const float*)out.ratios.p;
    d.zeros = has_zeros ? (const uint8_t*)out.zeros.p : nullptr;
    d.sz = has_zeros ? (const uint32_t*)out.sz.p : nullptr;
    d.K = K;
    d.N = N_dev;
    d.K_pad = K_pad;
    d.N_dev = N_dev;
    d.KG = KG;
    d.lgG = 0;
    while ((1 << d.lgG) < G) d.lgG++;
    d.wf = wf;
    return 0;
}

int validate_config(const layer_config* c) {
    if (!c) return fail(W4_EINVAL, "null config");
    if (c->hidden <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->ffn <= 0 || c->max_seq <= 0 ||
        c->max_batch <= 0)
        return fail(W4_EINVAL, "non-positive dimension in config");
    if (!(c->rms_eps >= 0.f) || !(c->rope_base > 0.f)) return fail(W4_EINVAL, "bad rms_eps or rope_base");
    if (c->head_dim != 64 && c->head_dim != 128) return fail(W4_EUNSUPPORTED, "head_dim must be 64 or 128");
    if (c->n_heads % c->n_kv_heads) return fail(W4_EUNSUPPORTED, "n_heads must be a multiple of n_kv_heads");
    if (c->n_heads / c->n_kv_heads > 8) return fail(W4_EUNSUPPORTED, "at most 8 query heads per kv head");
    if (c->weight_format < W4_WEIGHTS_INT4 || c->weight_format > W4_WEIGHTS_BF16)
        return fail(W4_EINVAL, "unknown weight_format %d", c->weight_format);
    // (the 8- and 16-bit formats keep one scale per column in groups of 128)
    const int G = c->weight_format == W4_WEIGHTS_INT4 ? c->group_size : 128;
    if (G != 32 && G != 64 && G != 128 && G != 256) return fail(W4_EUNSUPPORTED, "group_size must be 32, 64, 128 or 256");
    const int KP = std::max(64, G);
    if (c->hidden % 128 || c->hidden % KP) return fail(W4_EUNSUPPORTED, "hidden must be a multiple of 128 and of group_size");
    const int qd = c->n_heads * c->head_dim;
    if (qd % 128 || qd % KP) return fail(W4_EUNSUPPORTED, "n_heads*head_dim must be a multiple of 128 and of group_size");
    if (c->ffn % 8) return fail(W4_EUNSUPPORTED, "ffn must be a multiple of 8");
    if (c->max_batch > 64) return fail(W4_EUNSUPPORTED, "max_batch above 64");
    if (c->hidden > 16384 || round_up(c->ffn, std::max(128, KP)) > 65536) return fail(W4_EUNSUPPORTED, "hidden or ffn too large");
    return 0;
}

int check_device() {
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    hipDeviceProp_t prop;
    HIP_TRY(hipGetDeviceProperties(&prop, dev));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(W4_EUNSUPPORTED, "device %d is %s, this library is built for gfx950", dev, prop.gcnArchName);
    return 0;
}

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
int scratch_setup() {
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(W4_EUNSUPPORTED, "device index %d above %d", dev, kMaxDevices - 1);
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (g_scratch[dev]) return W4_OK;
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(W4_EHIP, "no device address for the scratch array");
    g_scratch[dev] = p;
    return W4_OK;
}

// ---- workspace plan
struct Carve {
    size_t off = 0;
    size_t take(size_t bytes) {
        const size_t o = off;
        off += (bytes + 255) / 256 * 256;
        return o;
    }
};

constexpr int kGemmCounters = 1024;     // split-K tiles of one GEMM (at most about one per CU)

struct PrefillWs {
    size_t xn1, q, attn, h, xn2, g, part, cnt, total;
    GemmPlan qkv, o, gu, down;
    AttnPrefillPlan at;
};
PrefillWs plan_prefill(const layer_s* L, int T, int hist) {
    const layer_config& c = L->cfg;
    const size_t qd = (size_t)c.n_heads * c.head_dim;
    Carve cv;
    PrefillWs w;
    w.qkv = gemm_w4_plan(T, L->qkv.d, L->num_cus);
    w.o = gemm_w4_plan(T, L->o.d, L->num_cus);
    w.gu = gemm_w4_plan(T, L->gu.d, L->num_cus);
    w.down = gemm_w4_plan(T, L->down.d, L->num_cus);
    w.at = attn_prefill_plan(T, hist, c.n_heads, c.n_kv_heads, c.head_dim, L->num_cus);
    w.xn1 = cv.take((size_t)T * c.hidden * 2);
    w.q = cv.take((size_t)T * qd * 2);
    w.attn = cv.take((size_t)T * qd * 2);
    w.h = cv.take((size_t)T * c.hidden * 4);
    w.xn2 = cv.take((size_t)T * c.hidden * 2);
    w.g = cv.take((size_t)T * L->F_pad * 2);
    // split-K partials of each GEMM and the attention chunk states, used one kernel at a time
    w.part = cv.take(std::max({w.qkv.part_bytes, w.o.part_bytes, w.gu.part_bytes, w.down.part_bytes, w.at.part_bound}));
    w.cnt = cv.take((size_t)kGemmCounters * 8);   // tagged split-K arrival counters
    w.total = cv.off;
    return w;
}

// keys per chunk of the separate-kernel decode attention (its split kernel
// stages one chunk of K and V in LDS)
int decode_chunk(int) { return 64; }

struct DecodeWs { size_t q, part, attn, h, g, xn, total; int chunk, nchunks; };
DecodeWs plan_decode(const layer_s* L, int B, int max_ctx) {
    const layer_config& c = L->cfg;
    const size_t qd = (size_t)c.n_heads * c.head_dim;
    DecodeWs w;
    w.chunk = decode_chunk(max_ctx);
    w.nchunks = (max_ctx + 1 + w.chunk - 1) / w.chunk;
    Carve cv;
    w.q = cv.take((size_t)B * qd * 2);
    w.part = cv.take((size_t)B * c.n_heads * w.nchunks * (c.head_dim + 2) * 4);
    w.attn = cv.take((size_t)B * qd * 2);
    w.h = cv.take((size_t)B * c.hidden * 4);
    w.g = cv.take((size_t)B * L->F_pad * 2);
    w.xn = cv.take((size_t)B * c.hidden * 2);
    w.total = cv.off;
    return w;
}

// ---- persistent decode plan
struct FusedPlan {
    bool ok = false;
    int nblocks = 0, chunk = 0, nchunk = 0, S_qkv = 1, S_o = 1, S_down = 1, ldx = 0, comb_per = 0, comb_lpv = 1;
    int slots = 0;                // gate/up column tiles of the busiest block
    int gam_lds = 1;              // RMSNorm weights in LDS
    size_t off_h = 0, off_red = 0, off_gam = 0, off_zero = 0, off_c64 = 0, lds_bytes = 0;
    size_t qkv_part = 0, apart = 0, A = 0, o_part = 0, g = 0, down_part = 0, total = 0;
};

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

// Column tiles of every product are owned by whole blocks; a product with
// fewer column tiles than blocks is also cut along k into S parts.
FusedPlan plan_fused(const layer_s* L, int B, int max_ctx, bool query_device) {
    FusedPlan p;
    const layer_config& c = L->cfg;
    if (B > 4 || L->decode_path == 1) return p;
    if (L->qkv.d.wf != WF_INT4) return p;                                    // 8- and 16-bit weights: separate kernels
    if (L->qkv.d.sz || L->o.d.sz || L->gu.d.sz || L->down.d.sz) return p;   // zero points: separate kernels
    if (c.group_size < 64) return p;                                         // groups of 32: separate kernels
    const int d = c.head_dim, qd = c.n_heads * d, H = c.hidden, r = c.n_heads / c.n_kv_heads;
    constexpr int MAXR = 8, NWAVE = 16;
    p.nblocks = 256;
    if (query_device) {
        int dev = 0, cus = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            return p;
        p.nblocks = cus;
    }
    const int P = p.nblocks;
    if (P > kMaxBlocks || r > MAXR || P != L->fused_blocks) return p;
    const int gu_pairs = L->gu.d.N_dev / 64;                                 // whole gate/up pairs per block
    p.slots = 2 * std::max(1, (gu_pairs + P - 1) / P);
    if (p.slots > 8) return p;
    p.S_qkv = L->S_qkv;
    p.S_o = L->S_o;
    p.S_down = L->S_down;
    // attention units: B * n_kv_heads * nchunk, about one per block; the
    // chunk shrinks (in steps of 32 keys) until the block's LDS fits
    const int per_group = std::max(1, P / (B * c.n_kv_heads));
    int ch = (max_ctx + 1 + per_group - 1) / per_group;
    ch = std::max(16, (ch + 15) / 16 * 16);
    ch = std::min(ch, decode_fused_max_chunk(d));
    const int kr_o = (L->o.d.K_pad / 64 + p.S_o - 1) / p.S_o * 64;
    const int kr_d = (L->down.d.K_pad / 64 + p.S_down - 1) / p.S_down * 64;
    p.ldx = std::max(std::max(H, kr_o), kr_d) + 8;
    const int maxb = B <= 1 ? 1 : 4;
    const size_t xs_bytes = (size_t)B * p.ldx * 2;
    // activation rows, then the GEMV's zero operand and correction table; the
    // attention phase reuses this region
    p.off_zero = align256(xs_bytes);
    p.off_c64 = p.off_zero + 256;
    const size_t gemv_bytes = p.off_c64 + (size_t)((p.ldx - 8) / 64) * 8 * 4;
    const int V = B * qd;
    p.comb_per = (((V + P - 1) / P) + 1) & ~1;
    const size_t comb_bytes = (size_t)p.comb_per * 2;
    // first with the RMSNorm weights in LDS, then (if no chunk fits) without
    const int ch0 = ch;
    for (int gl = 1; gl >= (B == 1 ? 1 : 0); gl--) {
        p.gam_lds = gl;
        for (ch = ch0;; ch = ch > 32 ? (ch - 1) / 32 * 32 : 16) {
            p.chunk = ch;
            p.nchunk = (max_ctx + 1 + ch - 1) / ch;
            p.off_h = align256(std::max(std::max(gemv_bytes, decode_fused_attn_bytes(ch, d)), comb_bytes));
            p.off_red = align256(p.off_h + (size_t)B * H * 4);
            p.off_gam = align256(p.off_red + (size_t)(NWAVE * p.slots * maxb * 32 + 8 + NWAVE * maxb + maxb * 32 + 2 * maxb) * 4);
            p.lds_bytes = p.off_gam + (gl ? (size_t)2 * H * 2 : 0);
            if (p.lds_bytes <= 160 * 1024 || ch == 16) break;
        }
        if (p.lds_bytes <= 160 * 1024) break;
    }
    if (p.lds_bytes > 160 * 1024) return p;
    p.comb_lpv = 1;
    while (p.comb_lpv < p.nchunk && p.comb_lpv < 64) p.comb_lpv *= 2;
    if (p.nchunk > 4 * p.comb_lpv) return p;
    if (query_device && decode_fused_blocks(d, B, p.lds_bytes) != p.nblocks) return p;
    Carve cv;
    p.qkv_part = cv.take((size_t)p.S_qkv * B * L->qkv.d.N_dev * 8);
    p.apart = cv.take((size_t)B * c.n_heads * p.nchunk * (d + 2) * 8);
    p.A = cv.take((size_t)B * qd / 2 * 8);
    p.o_part = cv.take((size_t)p.S_o * B * H * 8);
    p.g = cv.take((size_t)B * L->F_pad / 2 * 8);
    p.down_part = cv.take((size_t)p.S_down * B * H * 8);
    p.total = cv.off;
    p.ok = true;
    return p;
}

// Tag of a launch whose blocks hand data to each other through workspace
// words (the persistent decode, the split-K arrival counters): unique for
// 2^32 - 1 launches in the process and never 0 (a zeroed workspace holds no
// valid word).  The sequence starts at a point mixed from the clock and the
// process id, so a word that another process left in reused device memory
// matches a current tag only by chance (about 2^-32 per word).
uint32_t epoch_start() {
    uint64_t z = (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count() ^
                 ((uint64_t)getpid() << 32);
    z += 0x9E3779B97F4A7C15ull;   // splitmix64 finaliser
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return (uint32_t)(z ^ (z >> 31));
}

uint32_t next_epoch() {
    static std::atomic<uint32_t> ctr{epoch_start()};
    uint32_t e = ctr.fetch_add(1, std::memory_order_relaxed) + 1;
    if (e == 0) e = ctr.fetch_add(1, std::memory_order_relaxed) + 1;
    return e;
}

int gemv_ksplit(const DevLinear& W, int want_blocks, int B) {
    const int pairs = W.N_dev / 64, KB = W.K_pad / 64;
    int ks = std::max(1, std::min(KB, (want_blocks + pairs - 1) / pairs));
    // activation slice of B rows must fit the LDS budget (128 KB)
    while ((long long)B * ((KB + ks - 1) / ks) * 64 * 2 > 128 * 1024 && ks < KB) ks++;
    return ks;
}

// Event pair around kernel `k` of `stage` when it is the profiled one.
struct ProfScope {
    layer_s* L;
    int stage;
    bool on = false;
    hipStream_t st;
    // stage < 0: no timing (calls that must not allocate, even events)
    ProfScope(layer_s* L_, int stage_, int k, hipStream_t s) : L(L_), stage(stage_), st(s) {
        if (stage < 0) return;
        Profiler& p = L->prof;
        if (p.kernel[stage] == k && p.used[stage] < Profiler::kMax) {
            auto& ev = p.ev[stage];
            if ((int)ev.size() < 2 * (p.used[stage] + 1)) {
                hipEvent_t a, b;
                if (hipEventCreate(&a) != hipSuccess) return;
                if (hipEventCreate(&b) != hipSuccess) { (void)hipEventDestroy(a); return; }
                ev.push_back(a);
                ev.push_back(b);
            }
            on = hipEventRecord(ev[2 * p.used[stage]], st) == hipSuccess;
        }
    }
    ~ProfScope() {
        if (on) {
            Profiler& p = L->prof;
            if (hipEventRecord(p.ev[stage][2 * p.used[stage] + 1], st) == hipSuccess) p.used[stage]++;
        }
    }
};

EpiArgs base_epi(const layer_s* L) {
    EpiArgs e{};
    const layer_config& c = L->cfg;
    e.rope_cos = (const float*)L->rope_cos.p;
    e.rope_sin = (const float*)L->rope_sin.p;
    e.nq = c.n_heads;
    e.nkv = c.n_kv_heads;
    e.head_dim = c.head_dim;
    e.F_pad = L->F_pad;
    e.err = L->err;
    return e;
}

// The persistent decode launch for plan fp.  shared: the B rows are
// consecutive tokens of one sequence (prefill_kv with at most 4 tokens) with
// one cache, row b at context ctx_base + b; otherwise row b of a batch at
// context ctx_lens[b] in cache b.
int launch_fused(layer_s* L, const FusedPlan& fp, const float* x, const int32_t* pos, const int32_t* ctx_lens,
                 int ctx_base, bool shared, const float* attn_mask, int B, void* kc, void* vc, float* y, void* ws,
                 hipStream_t st) {
    const layer_config& c = L->cfg;
    char* base = (char*)ws;
    DecodeFusedArgs a{};
    a.qkv = L->qkv.d; a.o = L->o.d; a.gu = L->gu.d; a.down = L->down.d;
    a.attn_norm = (const uint16_t*)L->attn_norm.p;
    a.mlp_norm = (const uint16_t*)L->mlp_norm.p;
    a.eps = c.rms_eps;
    a.rope_cos = (const float*)L->rope_cos.p;
    a.rope_sin = (const float*)L->rope_sin.p;
    a.H = c.hidden; a.nq = c.n_heads; a.nkv = c.n_kv_heads; a.d = c.head_dim; a.F_pad = L->F_pad; a.B = B;
    a.x = x; a.pos = pos; a.ctx_lens = shared ? nullptr : ctx_lens; a.mask = attn_mask; a.max_seq = c.max_seq;
    a.ctx_base = ctx_base; a.shared = shared ? 1 : 0;
    a.k_cache = (uint16_t*)kc; a.v_cache = (uint16_t*)vc;
    a.sh = (long long)c.max_seq * c.head_dim; a.sb = shared ? 0 : a.sh * c.n_kv_heads;
    a.y = y;
    a.qkv_part = (uint64_t*)(base + fp.qkv_part);
    a.apart = (uint64_t*)(base + fp.apart);
    a.A = (uint64_t*)(base + fp.A);
    a.o_part = (uint64_t*)(base + fp.o_part);
    a.g = (uint64_t*)(base + fp.g);
    a.down_part = (uint64_t*)(base + fp.down_part);
    a.epoch = next_epoch();
    a.spin_max = L->spin_max;
    a.err = L->err;
    a.stamps = L->decode_trace ? L->stamps : nullptr;
    a.S_qkv = fp.S_qkv; a.S_o = fp.S_o; a.S_down = fp.S_down;
    a.comb_per = fp.comb_per; a.comb_lpv = fp.comb_lpv;
    a.slots = fp.slots;
    a.gam_lds = fp.gam_lds;
    a.chunk = fp.chunk; a.nchunk = fp.nchunk;
    a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)c.head_dim));
    a.nblocks = fp.nblocks;
    a.ldx = fp.ldx;
    a.off_h = fp.off_h;
    a.off_red = fp.off_red;
    a.off_gam = fp.off_gam;
    a.off_zero = fp.off_zero;
    a.off_c64 = fp.off_c64;
    a.lds_bytes = fp.lds_bytes;
    return launch_decode_fused(a, st);
}

// The decode as a sequence of kernels (GEMVs on up to 8 rows, split-KV
// attention, chunk merge).  shared: the B rows are consecutive tokens of one
// sequence with one cache (prefill / prefill_kv of at most 8 tokens), row b
// at context ctx_base + b: the q/k/v GEMV writes every row's new key and
// value before the attention kernel reads the cache.  ps_stage: the profiling
// stage the launches count for (2 decode, 0/1 prefill).
int run_decode_seq(layer_s* L, const float* x, const int32_t* pos, const int32_t* ctx_lens, int ctx_base, bool shared,
                   const float* attn_mask, int B, int max_ctx, void* kc, void* vc, float* y, void* ws,
                   size_t ws_bytes, hipStream_t st, int ps_stage) {
    const layer_config& c = L->cfg;
    const DecodeWs w = plan_decode(L, B, max_ctx);
    if (ws_bytes < w.total) return fail(W4_EWORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, w.total);
    char* base = (char*)ws;
    uint16_t* q = (uint16_t*)(base + w.q);
    float* part = (float*)(base + w.part);
    f16* attn = (f16*)(base + w.attn);
    float* h = (float*)(base + w.h);
    f16* g = (f16*)(base + w.g);
    const int H = c.hidden, d = c.head_dim, qd = c.n_heads * d;
    const long long sh = (long long)c.max_seq * d, sb = shared ? 0 : sh * c.n_kv_heads;
    int rc = 0;

    GemvArgs a1{};
    a1.W = L->qkv.d;
    a1.x_f32 = x;
    a1.gamma = (const uint16_t*)L->attn_norm.p;
    a1.eps = c.rms_eps;
    a1.B = B;
    a1.ksplit = 1;
    a1.ep = base_epi(L);
    a1.ep.q_out = q;
    a1.ep.k_cache = (uint16_t*)kc;
    a1.ep.v_cache = (uint16_t*)vc;
    a1.ep.cache_stride_b = sb;
    a1.ep.cache_stride_h = sh;
    a1.ep.pos = pos;
    a1.ep.slot_dev = shared ? nullptr : ctx_lens;
    a1.ep.slot_base = ctx_base;
    a1.copy_src = x;
    a1.copy_dst = h;
    a1.copy_n = B * H;
    // with 4 rows or more the rows are normalised once, not in every block
    const bool prenorm = B >= 4;
    f16* xn = (f16*)(base + w.xn);
    if (prenorm) {
        rc |= launch_rmsnorm(x, (const uint16_t*)L->attn_norm.p, c.rms_eps, B, H, xn, L->err, st);
        a1.x_f16 = xn;
        a1.ldx = H;
    }
    { ProfScope ps(L, ps_stage, ps_stage == 2 ? 0 : 1, st); rc |= launch_gemv_w4(EPI_QKV, !prenorm, a1, st); }

    AttnDecodeArgs ad{};
    ad.q = q;
    ad.k_cache = (const uint16_t*)kc;
    ad.v_cache = (const uint16_t*)vc;
    ad.stride_b = sb;
    ad.stride_h = sh;
    ad.ctx_lens = shared ? nullptr : ctx_lens;
    ad.ctx_base = ctx_base;
    ad.mask = attn_mask;
    ad.max_seq = c.max_seq;
    ad.part = part;
    ad.out = attn;
    ad.B = B;
    ad.nq = c.n_heads;
    ad.nkv = c.n_kv_heads;
    ad.d = d;
    ad.chunk = w.chunk;
    ad.nchunks = w.nchunks;
    ad.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d));
    ad.err = L->err;
    { ProfScope ps(L, ps_stage, ps_stage == 2 ? 1 : 2, st); rc |= launch_attn_decode(ad, st); }

    GemvArgs a2{};
    a2.W = L->o.d;
    a2.x_f16 = attn;
    a2.ldx = qd;
    a2.B = B;
    a2.ksplit = gemv_ksplit(L->o.d, 512, B);
    a2.ep = base_epi(L);
    a2.ep.out_f32 = h;
    { ProfScope ps(L, ps_stage, 3, st); rc |= launch_gemv_w4(EPI_RESID, false, a2, st); }

    GemvArgs a3{};
    a3.W = L->gu.d;
    a3.x_f32 = h;
    a3.gamma = (const uint16_t*)L->mlp_norm.p;
    a3.eps = c.rms_eps;
    a3.B = B;
    a3.ksplit = 1;
    a3.ep = base_epi(L);
    a3.ep.act_out = g;
    a3.copy_src = h;
    a3.copy_dst = y;
    a3.copy_n = B * H;
    if (prenorm) {
        rc |= launch_rmsnorm(h, (const uint16_t*)L->mlp_norm.p, c.rms_eps, B, H, xn, L->err, st);
        a3.x_f16 = xn;
        a3.ldx = H;
    }
    { ProfScope ps(L, ps_stage, ps_stage == 2 ? 4 : 5, st); rc |= launch_gemv_w4(EPI_SWIGLU, !prenorm, a3, st); }

    GemvArgs a4{};
    a4.W = L->down.d;
    a4.x_f16 = g;
    a4.ldx = L->F_pad;
    a4.B = B;
    a4.ksplit = gemv_ksplit(L->down.d, 512, B);
    a4.ep = base_epi(L);
    a4.ep.out_f32 = y;
    { ProfScope ps(L, ps_stage, ps_stage == 2 ? 5 : 6, st); rc |= launch_gemv_w4(EPI_RESID, false, a4, st); }
    if (rc) return fail(W4_EHIP, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
    return W4_OK;
}

// Prefill / prefill_kv of a few tokens runs on the decode kernels, the tokens
// as rows sharing one cache: up to 2 tokens (4 with decode path 2) as one
// persistent launch, up to 8 (decode path 0) as the decode kernel sequence;
// decode path 1 keeps every call on the prefill kernels.
FusedPlan small_prefill_plan(layer_s* L, int T, int hist) {
    if (!((L->decode_path == 0 && T <= 2) || (L->decode_path == 2 && T <= 4))) return FusedPlan{};
    return plan_fused(L, T, hist + T - 1, true);
}
bool small_prefill_seq(const layer_s* L, int T) { return L->decode_path == 0 && T <= 8; }

size_t prefill_ws_bytes(layer_s* L, int T, int hist) {
    size_t n = plan_prefill(L, T, hist).total;
    const FusedPlan fp = small_prefill_plan(L, T, hist);
    if (fp.ok) n = std::max(n, fp.total);
    else if (small_prefill_seq(L, T)) n = std::max(n, plan_decode(L, T, hist + T - 1).total);
    return n;
}

int run_prefill(layer_s* L, const float* x, const int32_t* pos, int T, int hist, void* kc, void* vc, float* y,
                void* ws, size_t ws_bytes, void* stream_) {
    if (!L) return fail(W4_EINVAL, "null layer");
    if (!x || !pos || !kc || !vc || !y || !ws) return fail(W4_EINVAL, "null pointer argument");
    if ((const void*)x == (const void*)y) return fail(W4_EINVAL, "x and y must not alias");
    const layer_config& c = L->cfg;
    if (T < 1 || hist < 0) return fail(W4_EINVAL, "T must be >= 1 and hist_len >= 0");
    if ((long long)hist + T > c.max_seq) return fail(W4_ECAPACITY, "hist_len + T = %lld exceeds max_seq %d", (long long)hist + T, c.max_seq);
    hipStream_t st = (hipStream_t)stream_;
    const int stage = hist > 0 ? 1 : 0;
    const FusedPlan fp = small_prefill_plan(L, T, hist);
    if (fp.ok) {
        if (ws_bytes < fp.total) return fail(W4_EWORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, fp.total);
        int rc;
        { ProfScope ps(L, stage, 7, st); rc = launch_fused(L, fp, x, pos, nullptr, hist, true, nullptr, T, kc, vc, y, ws, st); }
        if (rc) return fail(W4_EHIP, "persistent launch failed: %s", hipGetErrorString(hipGetLastError()));
        return W4_OK;
    }
    if (small_prefill_seq(L, T))
        return run_decode_seq(L, x, pos, nullptr, hist, true, nullptr, T, hist + T - 1, kc, vc, y, ws, ws_bytes, st, stage);
    const PrefillWs w = plan_prefill(L, T, hist);
    if (ws_bytes < w.total) return fail(W4_EWORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, w.total);
    char* base = (char*)ws;
    f16* xn1 = (f16*)(base + w.xn1);
    uint16_t* q = (uint16_t*)(base + w.q);
    f16* attn = (f16*)(base + w.attn);
    float* h = (float*)(base + w.h);
    f16* xn2 = (f16*)(base + w.xn2);
    f16* g = (f16*)(base + w.g);
    float* part = (float*)(base + w.part);
    unsigned long long* cnt = (unsigned long long*)(base + w.cnt);
    const int H = c.hidden, d = c.head_dim, qd = c.n_heads * d;
    for (const GemmPlan* gp : {&w.qkv, &w.o, &w.gu, &w.down})
        if (gp->S > 1 && gp->tiles > kGemmCounters) return fail(W4_EUNSUPPORTED, "split-K tile count above %d", kGemmCounters);

    int rc = 0;
    { ProfScope ps(L, stage, 0, st); rc |= launch_rmsnorm(x, (const uint16_t*)L->attn_norm.p, c.rms_eps, T, H, xn1, L->err, st); }
    EpiArgs e = base_epi(L);
    e.q_out = q;
    e.k_cache = (uint16_t*)kc;
    e.v_cache = (uint16_t*)vc;
    e.cache_stride_b = 0;
    e.cache_stride_h = (long long)c.max_seq * d;
    e.pos = pos;
    e.slot_base = hist;
    { ProfScope ps(L, stage, 1, st); rc |= launch_gemm_w4(EPI_QKV, xn1, H, L->qkv.d, e, w.qkv, T, part, cnt, next_epoch(), st); }
    AttnPrefillArgs aa{};
    aa.q = q;
    aa.k_cache = (const uint16_t*)kc;
    aa.v_cache = (const uint16_t*)vc;
    aa.cache_stride_h = (long long)c.max_seq * d;
    aa.out = attn;
    aa.T = T;
    aa.L = hist;
    aa.nq = c.n_heads;
    aa.nkv = c.n_kv_heads;
    aa.d = d;
    aa.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d));
    aa.part = part;
    aa.err = L->err;
    { ProfScope ps(L, stage, 2, st); rc |= launch_attn_prefill(aa, w.at, st); }
    EpiArgs eo = base_epi(L);
    eo.resid = x;
    eo.out_f32 = h;
    { ProfScope ps(L, stage, 3, st); rc |= launch_gemm_w4(EPI_RESID, attn, qd, L->o.d, eo, w.o, T, part, cnt, next_epoch(), st); }
    { ProfScope ps(L, stage, 4, st); rc |= launch_rmsnorm(h, (const uint16_t*)L->mlp_norm.p, c.rms_eps, T, H, xn2, L->err, st); }
    EpiArgs eg = base_epi(L);
    eg.act_out = g;
    { ProfScope ps(L, stage, 5, st); rc |= launch_gemm_w4(EPI_SWIGLU, xn2, H, L->gu.d, eg, w.gu, T, part, cnt, next_epoch(), st); }
    EpiArgs ed = base_epi(L);
    ed.resid = h;
    ed.out_f32 = y;
    { ProfScope ps(L, stage, 6, st); rc |= launch_gemm_w4(EPI_RESID, g, L->F_pad, L->down.d, ed, w.down, T, part, cnt, next_epoch(), st); }
    if (rc) return fail(W4_EHIP, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
    return W4_OK;
}

FusedPlan decode_fused_choice(layer_s* L, int B, int max_ctx);

// A checked decode call on workspace ws: the persistent launch or the kernel
// sequence.  ps_stage: 2 (the decode stage's kernel timing) or -1 (none).
int decode_run(layer_s* L, const float* x, const int32_t* pos, const int32_t* ctx_lens, int max_ctx,
               const float* attn_mask, int B, void* kc, void* vc, float* y, void* ws, size_t ws_bytes,
               hipStream_t st, int ps_stage) {
    const FusedPlan fp = decode_fused_choice(L, B, max_ctx);
    if (fp.ok) {
        if (ws_bytes < fp.total) return fail(W4_EWORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, fp.total);
        int rc;
        { ProfScope ps(L, ps_stage, 6, st); rc = launch_fused(L, fp, x, pos, ctx_lens, 0, false, attn_mask, B, kc, vc, y, ws, st); }
        if (rc) return fail(W4_EHIP, "persistent decode launch failed: %s", hipGetErrorString(hipGetLastError()));
        return W4_OK;
    }
    return run_decode_seq(L, x, pos, ctx_lens, 0, false, attn_mask, B, max_ctx, kc, vc, y, ws, ws_bytes, st, ps_stage);
}

// The persistent decode plan a decode call of B rows uses: forced by path 2,
// automatic for at most 2 rows (from 3 rows on the kernel sequence is the
// faster one); not ok means the kernel sequence.
FusedPlan decode_fused_choice(layer_s* L, int B, int max_ctx) {
    if (L->decode_path == 1 || (L->decode_path == 0 && B > 2)) return FusedPlan{};
    return plan_fused(L, B, max_ctx, true);
}

// Every check of a decode call of B rows up to context max_ctx that does not
// look at pointers, so a stack or model step can check all its layers
// before it enqueues the first kernel.
int decode_check(layer_s* L, int B, int max_ctx) {
    const layer_config& c = L->cfg;
    if (B < 1 || max_ctx < 0) return fail(W4_EINVAL, "B must be >= 1 and max_ctx >= 0");
    if (B > c.max_batch) return fail(W4_ECAPACITY, "B = %d exceeds max_batch %d", B, c.max_batch);
    if (B > 8) return fail(W4_EUNSUPPORTED, "decode batch above 8");
    if ((long long)max_ctx + 1 > c.max_seq)
        return fail(W4_ECAPACITY, "max_ctx + 1 = %lld exceeds max_seq %d", (long long)max_ctx + 1, c.max_seq);
    if (L->decode_path == 2 && !plan_fused(L, B, max_ctx, true).ok)
        return fail(W4_EUNSUPPORTED, "persistent decode not possible for this shape/batch");
    return W4_OK;
}

// The same for a prefill / prefill_kv call of T tokens after hist_len.
int prefill_check(layer_s* L, int T, int hist) {
    if (T < 1 || hist < 0) return fail(W4_EINVAL, "T must be >= 1 and hist_len >= 0");
    if ((long long)hist + T > L->cfg.max_seq)
        return fail(W4_ECAPACITY, "hist_len + T = %lld exceeds max_seq %d", (long long)hist + T, L->cfg.max_seq);
    return W4_OK;
}

}  // namespace

// =================================================================== C ABI

extern "C" {

const char* layer_last_error(void) { return g_err.c_str(); }

int kv_layout(const layer_config* cfg, int32_t batch, kv_desc* out) {
    if (!cfg || !out) return fail(W4_EINVAL, "null argument");
    if (batch < 1) return fail(W4_EINVAL, "batch must be >= 1");
    if (cfg->n_kv_heads <= 0 || cfg->max_seq <= 0 || cfg->head_dim <= 0) return fail(W4_EINVAL, "bad config");
    out->batch = batch;
    out->n_kv_heads = cfg->n_kv_heads;
    out->max_seq = cfg->max_seq;
    out->head_dim = cfg->head_dim;
    out->stride_s = cfg->head_dim;
    out->stride_h = (int64_t)cfg->max_seq * cfg->head_dim;
    out->stride_b = out->stride_h * cfg->n_kv_heads;
    out->bytes = (size_t)out->stride_b * batch * 2;
    return W4_OK;
}

int layer_create(const layer_config* cfg, const layer_weights_host* w, layer_t* out) {
    int rc;
    if ((rc = validate_config(cfg))) return rc;
    if (!w || !out) return fail(W4_EINVAL, "null argument");
    const qlinear_host* lins[7] = {&w->q, &w->k, &w->v, &w->o, &w->gate, &w->up, &w->down};
    const int fmt = cfg->weight_format;
    for (int i = 0; i < 7; i++) {
        const qlinear_host& q = *lins[i];
        const bool ok = fmt == W4_WEIGHTS_INT4 ? (q.qweight && q.scales)
                        : fmt == W4_WEIGHTS_INT8 ? (q.q8 && q.scales) : q.w16 != nullptr;
        if (!ok) return fail(W4_EINVAL, "null weight pointer (linear %d)", i);
    }
    if (!w->attn_norm || !w->mlp_norm) return fail(W4_EINVAL, "null norm weight");
    if ((rc = check_device())) return rc;
    if ((rc = scratch_setup())) return rc;
    const bool zq = w->q.zeros || w->k.zeros || w->v.zeros || w->o.zeros || w->gate.zeros || w->up.zeros || w->down.zeros;
    if (zq && !(w->q.zeros && w->k.zeros && w->v.zeros && w->o.zeros && w->gate.zeros && w->up.zeros && w->down.zeros))
        return fail(W4_EINVAL, "zero points must be given for all seven linears or for none");

    const layer_config& c = *cfg;
    const int H = c.hidden, d = c.head_dim, nq = c.n_heads, nkv = c.n_kv_heads, F = c.ffn;
    const int G = fmt == W4_WEIGHTS_INT4 ? c.group_size : 128;   // (8/16-bit: per column, groups of 128 on device)
    const int qd = nq * d, kvd = nkv * d;
    // K of every linear a multiple of 128 (and of G): the prefill GEMM takes
    // its k range in pairs of 64-k tiles
    const int F_pad = round_up(F, std::max(128, G));

    // scales must be finite; bf16 weights finite and below 4096 in magnitude
    // (the device holds 16 W in fp16 at half of the k positions)
    auto finite_scales = [&](const qlinear_host& q, int K, int N) {
        if (fmt == W4_WEIGHTS_BF16) {
            const size_t n = (size_t)K * N;
            for (size_t i = 0; i < n; i++) {
                const uint16_t b = q.w16[i];
                if (((b >> 7) & 0xFF) == 0xFF || !(std::fabs(bf16_value(b)) < 4096.0)) return false;
            }
            return true;
        }
        const size_t n = (size_t)(fmt == W4_WEIGHTS_INT8 ? 1 : (K + G - 1) / G) * N;
        for (size_t i = 0; i < n; i++)
            if (((q.scales[i] >> 10) & 0x1F) == 0x1F) return false;
        return true;
    };
    auto host_lin = [&](const qlinear_host& q, int K, int N) {
        HostLin h{q.qweight, q.scales, q.zeros, K, N};
        h.fmt = fmt;
        h.q8 = q.q8;
        h.w16 = q.w16;
        return h;
    };
    HostLin hq = host_lin(w->q, H, qd), hk = host_lin(w->k, H, kvd), hv = host_lin(w->v, H, kvd),
            ho = host_lin(w->o, qd, H), hg = host_lin(w->gate, H, F), hu = host_lin(w->up, H, F),
            hd = host_lin(w->down, F, H);
    const HostLin* all[7] = {&hq, &hk, &hv, &ho, &hg, &hu, &hd};
    for (int i = 0; i < 7; i++)
        if (!finite_scales(*lins[i], all[i]->K, all[i]->N))
            return fail(W4_EINVAL, fmt == W4_WEIGHTS_BF16 ? "bf16 weight not finite or not below 4096 in linear %d"
                                                           : "non-finite scale in linear %d", i);

    layer_s* L = new layer_s();
    L->cfg = c;
    L->F_pad = F_pad;
    (void)hipGetDevice(&L->device);

    // fused q|k|v with the RoPE block order inside each head
    std::vector<ColSrc> cq(qd + 2 * kvd);
    std::vector<int32_t> mq(qd), mk(kvd), mv(kvd);
    for (int nd = 0; nd < qd + 2 * kvd; nd++) {
        int local = nd;
        const HostLin* src = &hq;
        std::vector<int32_t>* map = &mq;
        if (local >= qd + kvd) { local -= qd + kvd; src = &hv; map = &mv; }
        else if (local >= qd) { local -= qd; src = &hk; map = &mk; }
        const int head = local / d, p = (local % d) / 32;
        const int dim = 32 * rope_block(p, d) + local % 32;
        cq[nd] = ColSrc{src, head * d + dim};
        (*map)[head * d + dim] = nd;
    }
    std::vector<ColSrc> co(H), cd(H);
    std::vector<int32_t> mo(H), md(H);
    for (int n = 0; n < H; n++) { co[n] = ColSrc{&ho, n}; cd[n] = ColSrc{&hd, n}; mo[n] = n; md[n] = n; }
    std::vector<ColSrc> cgu(2 * F_pad);
    std::vector<int32_t> mg(F), mu(F);
    for (int nd = 0; nd < 2 * F_pad; nd++) {
        const int j2 = nd / 32, j = j2 / 2, which = j2 % 2, f = 32 * j + nd % 32;
        if (f < F) {
            cgu[nd] = ColSrc{which ? &hu : &hg, f};
            (which ? mu : mg)[f] = nd;
        } else {
            cgu[nd] = ColSrc{nullptr, 0};
        }
    }
    if ((rc = build_linear(L->qkv, cq, H, H, G, zq, fmt)) || (rc = build_linear(L->o, co, qd, qd, G, zq, fmt)) ||
        (rc = build_linear(L->gu, cgu, H, H, G, zq, fmt)) || (rc = build_linear(L->down, cd, F, F_pad, G, zq, fmt)) ||
        (rc = upload(L->qkv.colmap_a, mq.data(), mq.size() * 4)) || (rc = upload(L->qkv.colmap_b, mk.data(), mk.size() * 4)) ||
        (rc = upload(L->qkv.colmap_c, mv.data(), mv.size() * 4)) || (rc = upload(L->o.colmap_a, mo.data(), mo.size() * 4)) ||
        (rc = upload(L->gu.colmap_a, mg.data(), mg.size() * 4)) || (rc = upload(L->gu.colmap_b, mu.data(), mu.size() * 4)) ||
        (rc = upload(L->down.colmap_a, md.data(), md.size() * 4)) ||
        (rc = upload(L->attn_norm, w->attn_norm, (size_t)H * 2)) || (rc = upload(L->mlp_norm, w->mlp_norm, (size_t)H * 2))) {
        delete L;
        return rc;
    }
    // RoPE cos/sin table, computed in double (Sec. 4.6.2)
    std::vector<float> tc((size_t)c.max_seq * (d / 2)), ts(tc.size());
    for (int p = 0; p < c.max_seq; p++)
        for (int i = 0; i < d / 2; i++) {
            const double ang = (double)p * std::pow((double)c.rope_base, -2.0 * i / d);
            tc[(size_t)p * (d / 2) + i] = (float)std::cos(ang);
            ts[(size_t)p * (d / 2) + i] = (float)std::sin(ang);
        }
    if ((rc = upload(L->rope_cos, tc.data(), tc.size() * 4)) || (rc = upload(L->rope_sin, ts.data(), ts.size() * 4))) {
        delete L;
        return rc;
    }
    {
        // [0]: error flag; from byte 64: stamps (8 + 32 * max blocks words of 8 bytes)
        const size_t bytes = 64 + (size_t)kStampWords * 8;
        std::vector<unsigned char> zero(bytes, 0);
        if ((rc = upload(L->sync, zero.data(), bytes))) { delete L; return rc; }
        L->err = (int*)L->sync.p;
        L->stamps = (unsigned long long*)((char*)L->sync.p + 64);
    }
    // work split of the persistent decode: one block per CU; a product with
    // fewer column tiles than blocks is also cut along k (at most 2 parts)
    {
        int dev = 0, cus = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
            L->num_cus = cus;
        if (cus > 0 && cus <= kMaxBlocks) {
            auto parts = [&](const DevLinear& W) {
                const int nt = W.N_dev / 32, kb = W.K_pad / 64;
                return std::max(1, std::min(std::min(2, kb), cus / nt));
            };
            if (L->qkv.d.N_dev / 32 <= cus && L->o.d.N_dev / 32 <= cus && L->down.d.N_dev / 32 <= cus) {
                L->S_qkv = parts(L->qkv.d);
                // o_proj stays whole: its sums go to every block (the RMSNorm of
                // h needs all of them), and a second k part doubles that hand-off
                L->S_o = 1;
                L->S_down = parts(L->down.d);
                L->fused_blocks = cus;
            }
        }
    }
    *out = L;
    return W4_OK;
}

int layer_destroy(layer_t layer) {
    if (!layer) return W4_OK;
    (void)hipDeviceSynchronize();
    delete layer;
    return W4_OK;
}

size_t layer_workspace_size(layer_t L, int32_t stage, int32_t batch, int32_t T, int32_t max_ctx) {
    if (!L) return 0;
    if (stage == 0 || stage == 1) {
        if (T < 1 || max_ctx < 0) return 0;
        return prefill_ws_bytes(L, T, stage == 1 ? max_ctx : 0);
    }
    if (stage == 2) {
        if (batch < 1 || max_ctx < 0) return 0;
        size_t n = plan_decode(L, batch, max_ctx).total;
        const FusedPlan fp = plan_fused(L, batch, max_ctx, true);
        if (fp.ok) n = std::max(n, fp.total);
        return n;
    }
    return 0;
}

int layer_prefill(layer_t L, const float* x, const int32_t* pos, int32_t T, void* kc, void* vc, float* y, void* ws,
                  size_t ws_bytes, void* stream) {
    return run_prefill(L, x, pos, T, 0, kc, vc, y, ws, ws_bytes, stream);
}

int layer_prefill_kv(layer_t L, const float* x, const int32_t* pos, int32_t T, int32_t hist_len, void* kc, void* vc,
                     float* y, void* ws, size_t ws_bytes, void* stream) {
    return run_prefill(L, x, pos, T, hist_len, kc, vc, y, ws, ws_bytes, stream);
}

size_t layer_prefill_chunked_workspace_size(layer_t L, int32_t T, int32_t chunk) {
    if (!L || T < 1 || chunk < 1) return 0;
    size_t n = 0;
    for (int s = 0; s < T; s += chunk) n = std::max(n, prefill_ws_bytes(L, std::min(chunk, T - s), s));
    return n;
}

int layer_prefill_chunked(layer_t L, const float* x, const int32_t* pos, int32_t T, int32_t chunk, void* kc,
                          void* vc, float* y, void* ws, size_t ws_bytes, void* stream) {
    if (!L) return fail(W4_EINVAL, "null layer");
    if (!x || !pos || !kc || !vc || !y || !ws) return fail(W4_EINVAL, "null pointer argument");
    if (T < 1 || chunk < 1) return fail(W4_EINVAL, "T and chunk must be >= 1");
    if (T > L->cfg.max_seq) return fail(W4_ECAPACITY, "T = %d exceeds max_seq %d", T, L->cfg.max_seq);
    const size_t need = layer_prefill_chunked_workspace_size(L, T, chunk);
    if (ws_bytes < need) return fail(W4_EWORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
    const size_t H = (size_t)L->cfg.hidden;
    for (int s = 0; s < T; s += chunk) {
        const int n = std::min(chunk, T - s);
        const int rc = run_prefill(L, x + (size_t)s * H, pos + s, n, s, kc, vc, y + (size_t)s * H, ws, ws_bytes, stream);
        if (rc) return rc;
    }
    return W4_OK;
}

int layer_decode(layer_t L, const float* x, const int32_t* pos, const int32_t* ctx_lens, int32_t max_ctx,
                 const float* attn_mask, int32_t B, void* kc, void* vc, float* y, void* ws, size_t ws_bytes,
                 void* stream) {
    if (!L) return fail(W4_EINVAL, "null layer");
    if (!x || !pos || !ctx_lens || !kc || !vc || !y || !ws) return fail(W4_EINVAL, "null pointer argument");
    if ((const void*)x == (const void*)y) return fail(W4_EINVAL, "x and y must not alias");
    int rc;
    if ((rc = decode_check(L, B, max_ctx))) return rc;
    return decode_run(L, x, pos, ctx_lens, max_ctx, attn_mask, B, kc, vc, y, ws, ws_bytes, (hipStream_t)stream, 2);
}

int layer_decode_noalloc(layer_t L, const float* x, const int32_t* pos, const int32_t* ctx_lens, int32_t max_ctx,
                         const float* attn_mask, int32_t B, void* kc, void* vc, float* y, void* stream) {
    if (!L) return fail(W4_EINVAL, "null layer");
    if (!x || !pos || !ctx_lens || !kc || !vc || !y) return fail(W4_EINVAL, "null pointer argument");
    if ((const void*)x == (const void*)y) return fail(W4_EINVAL, "x and y must not alias");
    int rc;
    if ((rc = decode_check(L, B, max_ctx))) return rc;
    if (L->device < 0 || L->device >= kMaxDevices || !g_scratch[L->device])
        return fail(W4_EHIP, "scratch array not set up on device %d", L->device);
    const size_t need = layer_workspace_size(L, 2, B, 1, max_ctx);
    if (need == 0 || need > kScratchBytes)
        return fail(W4_EWORKSPACE, "decode of B = %d at context %d needs %zu bytes of scratch; the static scratch "
                    "array holds %zu", B, max_ctx, need, kScratchBytes);
    return decode_run(L, x, pos, ctx_lens, max_ctx, attn_mask, B, kc, vc, y, g_scratch[L->device], kScratchBytes,
                      (hipStream_t)stream, -1);
}

size_t layer_decode_noalloc_max_bytes(void) { return kScratchBytes; }

int kv_append(const kv_desc* desc, void* kc, void* vc, const void* k_new, const void* v_new, int32_t B, int32_t T,
              const int32_t* slot_start, void* stream) {
    if (!desc || !kc || !vc || !k_new || !v_new || !slot_start) return fail(W4_EINVAL, "null argument");
    if (B < 1 || T < 1) return fail(W4_EINVAL, "B and T must be >= 1");
    if (desc->head_dim % 8 || desc->head_dim <= 0 || desc->n_kv_heads <= 0 || desc->stride_s != desc->head_dim)
        return fail(W4_EINVAL, "bad kv_desc");
    if (B > desc->batch || B > 64) return fail(W4_ECAPACITY, "B = %d exceeds the cache batch", B);
    for (int b = 0; b < B; b++)
        if (slot_start[b] < 0 || (long long)slot_start[b] + T > desc->max_seq)
            return fail(W4_ECAPACITY, "slots %d..%d of sequence %d outside max_seq %d", slot_start[b], slot_start[b] + T - 1, b, desc->max_seq);
    if (launch_kv_append((uint16_t*)kc, (uint16_t*)vc, (const uint16_t*)k_new, (const uint16_t*)v_new, B, T,
                         desc->n_kv_heads, desc->head_dim, desc->stride_b, desc->stride_h, slot_start,
                         (hipStream_t)stream))
        return fail(W4_EHIP, "kv_append launch failed: %s", hipGetErrorString(hipGetLastError()));
    return W4_OK;
}

int layer_debug_dequant(layer_t L, int32_t which, float* out, void* stream) {
    if (!L || !out) return fail(W4_EINVAL, "null argument");
    if (which < 0 || which > 6) return fail(W4_EINVAL, "which must be 0..6");
    const layer_config& c = L->cfg;
    const int H = c.hidden, qd = c.n_heads * c.head_dim, kvd = c.n_kv_heads * c.head_dim, F = c.ffn;
    const DevLinearOwned* dl;
    const void* map;
    int K, N;
    switch (which) {
        case 0: dl = &L->qkv; map = L->qkv.colmap_a.p; K = H; N = qd; break;
        case 1: dl = &L->qkv; map = L->qkv.colmap_b.p; K = H; N = kvd; break;
        case 2: dl = &L->qkv; map = L->qkv.colmap_c.p; K = H; N = kvd; break;
        case 3: dl = &L->o; map = L->o.colmap_a.p; K = qd; N = H; break;
        case 4: dl = &L->gu; map = L->gu.colmap_a.p; K = H; N = F; break;
        case 5: dl = &L->gu; map = L->gu.colmap_b.p; K = H; N = F; break;
        default: dl = &L->down; map = L->down.colmap_a.p; K = F; N = H; break;
    }
    if (launch_debug_dequant(dl->d, (const int32_t*)map, K, N, out, (hipStream_t)stream))
        return fail(W4_EHIP, "debug dequant launch failed: %s", hipGetErrorString(hipGetLastError()));
    return W4_OK;
}

// ---------------------------------------------------------------- stacks

// Activations between layers: two fp32 [rows][hidden] buffers after the
// layers' own workspace (256-byte aligned).
static size_t stack_act_offset(size_t layer_ws) { return (layer_ws + 255) / 256 * 256; }

static int check_stack(const layer_t* layers, int32_t n) {
    if (!layers || n < 1) return fail(W4_EINVAL, "null layer list or n_layers < 1");
    for (int i = 0; i < n; i++) {
        if (!layers[i]) return fail(W4_EINVAL, "null layer %d", i);
        if (layers[i]->cfg.hidden != layers[0]->cfg.hidden) return fail(W4_EINVAL, "layer %d: hidden differs", i);
    }
    return W4_OK;
}

size_t stack_workspace_size(const layer_t* layers, int32_t n, int32_t stage, int32_t batch, int32_t T,
                            int32_t max_ctx) {
    if (check_stack(layers, n)) return 0;
    size_t w = 0;
    for (int i = 0; i < n; i++) {
        const size_t wi = layer_workspace_size(layers[i], stage, batch, T, max_ctx);
        if (wi == 0) return 0;
        w = std::max(w, wi);
    }
    const size_t rows = stage == 2 ? (size_t)batch : (size_t)T;
    return stack_act_offset(w) + 2 * rows * layers[0]->cfg.hidden * sizeof(float);
}

int stack_prefill(const layer_t* layers, int32_t n, const float* x, const int32_t* pos, int32_t T, int32_t hist_len,
                  void* const* k_caches, void* const* v_caches, float* y, void* ws, size_t ws_bytes, void* stream) {
    int rc;
    if ((rc = check_stack(layers, n))) return rc;
    if (!x || !y || !ws || !k_caches || !v_caches) return fail(W4_EINVAL, "null pointer argument");
    if ((const void*)x == (const void*)y) return fail(W4_EINVAL, "x and y must not alias");
    for (int i = 0; i < n; i++)
        if ((rc = prefill_check(layers[i], T, hist_len))) return rc;
    const size_t need = stack_workspace_size(layers, n, hist_len > 0 ? 1 : 0, 1, T, hist_len);
    if (need == 0 || ws_bytes < need) return fail(W4_EWORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
    const size_t act = stack_act_offset(need - 2 * (size_t)T * layers[0]->cfg.hidden * sizeof(float));
    float* buf[2] = {(float*)((char*)ws + act), (float*)((char*)ws + act) + (size_t)T * layers[0]->cfg.hidden};
    const float* in = x;
    for (int i = 0; i < n; i++) {
        float* out = i == n - 1 ? y : buf[i & 1];
        if ((rc = run_prefill(layers[i], in, pos, T, hist_len, k_caches[i], v_caches[i], out, ws, act, stream))) return rc;
        in = out;
    }
    return W4_OK;
}

int stack_decode(const layer_t* layers, int32_t n, const float* x, const int32_t* pos, const int32_t* ctx_lens,
                 int32_t max_ctx, const float* attn_mask, int32_t B, void* const* k_caches, void* const* v_caches,
                 float* y, void* ws, size_t ws_bytes, void* stream) {
    int rc;
    if ((rc = check_stack(layers, n))) return rc;
    if (!x || !y || !ws || !k_caches || !v_caches) return fail(W4_EINVAL, "null pointer argument");
    if ((const void*)x == (const void*)y) return fail(W4_EINVAL, "x and y must not alias");
    for (int i = 0; i < n; i++)
        if ((rc = decode_check(layers[i], B, max_ctx))) return rc;
    const size_t need = stack_workspace_size(layers, n, 2, B, 1, max_ctx);
    if (need == 0 || ws_bytes < need) return fail(W4_EWORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
    const size_t act = stack_act_offset(need - 2 * (size_t)B * layers[0]->cfg.hidden * sizeof(float));
    float* buf[2] = {(float*)((char*)ws + act), (float*)((char*)ws + act) + (size_t)B * layers[0]->cfg.hidden};
    const float* in = x;
    for (int i = 0; i < n; i++) {
        float* out = i == n - 1 ? y : buf[i & 1];
        if ((rc = layer_decode(layers[i], in, pos, ctx_lens, max_ctx, attn_mask, B, k_caches[i], v_caches[i], out, ws,
                               act, stream)))
            return rc;
        in = out;
    }
    return W4_OK;
}

int layer_error(layer_t L, int32_t* flag) {
    if (!L || !flag) return fail(W4_EINVAL, "null argument");
    int v = 0;
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(hipMemcpy(&v, L->err, sizeof v, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemset(L->err, 0, sizeof v));
    HIP_TRY(hipDeviceSynchronize());
    *flag = v;
    return W4_OK;
}

int layer_decode_phase_times(layer_t L, float* us_out, int32_t* error_flag) {
    if (!L || !us_out) return fail(W4_EINVAL, "null argument");
    std::vector<unsigned long long> ts(kStampWords);
    int err = 0;
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(hipMemcpy(ts.data(), L->stamps, ts.size() * 8, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(&err, L->err, sizeof err, hipMemcpyDeviceToHost));
    int khz = 0;
    HIP_TRY(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, L->device));
    const int nb = (int)std::min<unsigned long long>(ts[1], kMaxBlocks);
    // end of phase i: the last block to finish it
    unsigned long long prev = ts[0];
    for (int i = 0; i < 5; i++) {
        unsigned long long e = prev;
        for (int b = 0; b < nb; b++) e = std::max(e, ts[8 + (size_t)i * nb + b]);
        us_out[i] = khz > 0 ? (float)((double)(e - prev) * 1000.0 / khz) : 0.f;
        prev = e;
    }
    if (error_flag) *error_flag = err;
    return W4_OK;
}

int layer_debug_decode_stamps(layer_t L, uint64_t* out, int32_t n) {
    if (!L || !out || n < 0) return fail(W4_EINVAL, "bad argument");
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(hipMemcpy(out, L->stamps, (size_t)std::min(n, kStampWords) * 8, hipMemcpyDeviceToHost));
    return W4_OK;
}

int layer_set_decode_path(layer_t L, int32_t path) {
    if (!L) return fail(W4_EINVAL, "null layer");
    if (path < 0 || path > 2) return fail(W4_EINVAL, "path must be 0, 1 or 2");
    L->decode_path = path;
    return W4_OK;
}

int layer_set_decode_spin_limit(layer_t L, int32_t polls) {
    if (!L) return fail(W4_EINVAL, "null layer");
    if (polls < 0) return fail(W4_EINVAL, "polls must be >= 0");
    L->spin_max = polls == 0 ? kSpinDefault : polls;
    return W4_OK;
}

int layer_set_decode_trace(layer_t L, int32_t on) {
    if (!L) return fail(W4_EINVAL, "null layer");
    L->decode_trace = on != 0;
    return W4_OK;
}

int layer_profile_kernel(layer_t L, int32_t stage, int32_t kernel) {
    if (!L) return fail(W4_EINVAL, "null layer");
    if (stage < 0 || stage > 2) return fail(W4_EINVAL, "stage must be 0..2");
    L->prof.kernel[stage] = kernel < 0 ? -1 : kernel;
    if (kernel >= 0 && kernel != L->prof.recorded[stage]) {
        L->prof.used[stage] = 0;
        L->prof.recorded[stage] = kernel;
    }
    return W4_OK;
}

int layer_profile_read(layer_t L, int32_t stage, float* total_ms, int32_t* launches) {
    if (!L || !total_ms || !launches) return fail(W4_EINVAL, "null argument");
    if (stage < 0 || stage > 2) return fail(W4_EINVAL, "stage must be 0..2");
    Profiler& p = L->prof;
    double tot = 0.0;
    for (int i = 0; i < p.used[stage]; i++) {
        HIP_TRY(hipEventSynchronize(p.ev[stage][2 * i + 1]));
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, p.ev[stage][2 * i], p.ev[stage][2 * i + 1]));
        tot += ms;
    }
    *total_ms = (float)tot;
    *launches = p.used[stage];
    p.used[stage] = 0;
    return W4_OK;
}

}  // extern "C"

// ---------------------------------------------------------------- model ends

struct lm_s {
    lm_config cfg{};
    DevLinearOwned head;
    DevBuf embed, final_norm, zeros, err;
    int device = 0;
};

namespace {

constexpr int kLmRows = 8;   // rows per launch of the head's GEMV

size_t lm_ws_layout(const lm_s* M, int B, size_t* off_pv, size_t* off_pi) {
    const size_t a = 256;
    const size_t xn = ((size_t)B * M->cfg.hidden * 2 + a - 1) / a * a;
    const size_t pairs = (size_t)B * argmax_blocks(M->cfg.vocab);
    const size_t pv = (pairs * 4 + a - 1) / a * a;
    if (off_pv) *off_pv = xn;
    if (off_pi) *off_pi = xn + pv;
    return xn + pv + (pairs * 4 + a - 1) / a * a;
}

}  // namespace

extern "C" {

int lm_create(const lm_config* cfg, const lm_weights_host* w, lm_t* out) {
    if (!cfg || !w || !out) return fail(W4_EINVAL, "null argument");
    *out = nullptr;
    const lm_config c = *cfg;
    const int G = c.group_size;
    if (c.vocab <= 0 || c.hidden <= 0 || c.max_batch <= 0 || !(c.rms_eps >= 0.f))
        return fail(W4_EINVAL, "non-positive dimension or bad rms_eps in config");
    if (c.vocab % 64) return fail(W4_EUNSUPPORTED, "vocab must be a multiple of 64");
    if (G != 32 && G != 64 && G != 128 && G != 256) return fail(W4_EUNSUPPORTED, "group_size must be 32, 64, 128 or 256");
    if (c.hidden % 128 || c.hidden % G || c.hidden > 7680)
        return fail(W4_EUNSUPPORTED, "hidden must be a multiple of 128 and of group_size, at most 7680");
    if (c.max_batch > 64) return fail(W4_EUNSUPPORTED, "max_batch must be at most 64");
    if (!w->embed || !w->final_norm || !w->head.qweight || !w->head.scales) return fail(W4_EINVAL, "null weight");
    const int H = c.hidden, V = c.vocab, KG = H / G;
    for (size_t i = 0; i < (size_t)KG * V; i++)
        if ((w->head.scales[i] & 0x7C00u) == 0x7C00u) return fail(W4_EINVAL, "non-finite scale in the LM head");
    if (w->head.zeros)
        for (size_t i = 0; i < (size_t)KG * V; i++)
            if (w->head.zeros[i] > 15) return fail(W4_EINVAL, "zero point above 15 in the LM head");

    lm_s* M = new lm_s();
    M->cfg = c;
    (void)hipGetDevice(&M->device);
    const HostLin hl{w->head.qweight, w->head.scales, w->head.zeros, H, V};
    std::vector<ColSrc> cols(V);
    for (int n = 0; n < V; n++) cols[n] = ColSrc{&hl, n};
    int rc = build_linear(M->head, cols, H, H, G, w->head.zeros != nullptr);
    if (!rc) rc = upload(M->embed, w->embed, (size_t)V * H * 2);
    if (!rc) rc = upload(M->final_norm, w->final_norm, (size_t)H * 2);
    if (!rc) {
        // all-zero residual rows: the head's GEMV stores 0 + sum
        const size_t zb = (size_t)kLmRows * V * 4;
        if (hipMalloc(&M->zeros.p, zb) != hipSuccess || hipMemset(M->zeros.p, 0, zb) != hipSuccess ||
            hipMalloc(&M->err.p, 4) != hipSuccess || hipMemset(M->err.p, 0, 4) != hipSuccess ||
            hipDeviceSynchronize() != hipSuccess)
            rc = fail(W4_EHIP, "device allocation failed");
    }
    if (rc) {
        delete M;
        return rc;
    }
    *out = M;
    return W4_OK;
}

int lm_destroy(lm_t lm) {
    if (!lm) return fail(W4_EINVAL, "null handle");
    delete lm;
    return W4_OK;
}

int lm_embed(lm_t M, const int32_t* tokens, int32_t B, float* x, void* stream) {
    if (!M || !tokens || !x) return fail(W4_EINVAL, "null argument");
    if (B < 1) return fail(W4_EINVAL, "B must be positive");
    if (launch_embed((const uint16_t*)M->embed.p, tokens, M->cfg.vocab, M->cfg.hidden, B, x, (int*)M->err.p,
                     (hipStream_t)stream))
        return fail(W4_EHIP, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
    return W4_OK;
}

size_t lm_head_workspace_size(lm_t M, int32_t B) {
    if (!M || B < 1 || B > M->cfg.max_batch) return 0;
    return lm_ws_layout(M, B, nullptr, nullptr);
}

int lm_head(lm_t M, const float* x, int32_t B, float* logits, int32_t* next_tokens, void* ws, size_t ws_bytes,
            void* stream) {
    if (!M || !x || !logits) return fail(W4_EINVAL, "null argument");
    if (B < 1) return fail(W4_EINVAL, "B must be positive");
    if (B > M->cfg.max_batch) return fail(W4_ECAPACITY, "B %d > max_batch %d", B, M->cfg.max_batch);
    size_t off_pv = 0, off_pi = 0;
    const size_t need = lm_ws_layout(M, B, &off_pv, &off_pi);
    if (!ws || ws_bytes < need) return fail(W4_EWORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, need);
    hipStream_t st = (hipStream_t)stream;
    const lm_config& c = M->cfg;
    const int H = c.hidden, V = c.vocab;
    f16* xn = (f16*)ws;
    int rc = launch_rmsnorm(x, (const uint16_t*)M->final_norm.p, c.rms_eps, B, H, xn, (int*)M->err.p, st);
    for (int r0 = 0; r0 < B && !rc; r0 += kLmRows) {
        GemvArgs a{};
        a.W = M->head.d;
        a.x_f16 = xn + (size_t)r0 * H;
        a.ldx = H;
        a.B = std::min(kLmRows, B - r0);
        a.ksplit = 1;
        a.ep.resid = (const float*)M->zeros.p;
        a.ep.out_f32 = logits + (size_t)r0 * V;
        rc = launch_gemv_w4(EPI_RESID, false, a, st);
    }
    if (!rc && next_tokens)
        rc = launch_argmax(logits, B, V, (float*)((char*)ws + off_pv), (int*)((char*)ws + off_pi), next_tokens, st);
    if (rc) return fail(W4_EHIP, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
    return W4_OK;
}

int lm_error(lm_t M, int32_t* flag) {
    if (!M || !flag) return fail(W4_EINVAL, "null argument");
    int v = 0;
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(hipMemcpy(&v, M->err.p, 4, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemset(M->err.p, 0, 4));
    HIP_TRY(hipDeviceSynchronize());
    *flag = v;
    return W4_OK;
}

// ---------------------------------------------------------------- runtime loop step

namespace {
size_t model_act_bytes(int B, int H) { return ((size_t)B * H * 4 + 255) / 256 * 256; }
// every layer can decode B sequences at a context up to max_ctx (the checks
// of a decode call: capacity, the batch limit, a forced persistent path)
int model_check(const layer_t* layers, int n, int B, int max_ctx) {
    for (int i = 0; i < n; i++) {
        if (!layers[i]) return fail(W4_EINVAL, "null layer %d", i);
        const int rc = decode_check(layers[i], B, max_ctx);
        if (rc) return rc;
    }
    return W4_OK;
}
}

size_t model_decode_workspace_size(const layer_t* layers, int32_t n_layers, lm_t lm, int32_t B, int32_t max_ctx) {
    if (!layers || n_layers < 1 || !lm || !layers[0] || layers[0]->cfg.hidden != lm->cfg.hidden) return 0;
    if (B < 1 || max_ctx < 0 || model_check(layers, n_layers, B, max_ctx) != W4_OK) return 0;
    const size_t st = stack_workspace_size(layers, n_layers, 2, B, 1, max_ctx);
    const size_t hd = lm_head_workspace_size(lm, B);
    if (!st || !hd) return 0;
    return 2 * model_act_bytes(B, lm->cfg.hidden) + std::max(st, hd);
}

int model_decode_greedy(const layer_t* layers, int32_t n_layers, lm_t lm, const int32_t* tokens, const int32_t* pos,
                        const int32_t* ctx_lens, int32_t max_ctx, int32_t B, void* const* k_caches,
                        void* const* v_caches, float* logits, int32_t* next_tokens, void* ws, size_t ws_bytes,
                        void* stream) {
    if (!layers || n_layers < 1 || !lm || !tokens || !pos || !ctx_lens || !k_caches || !v_caches || !logits ||
        !next_tokens)
        return fail(W4_EINVAL, "null pointer argument");
    for (int i = 0; i < n_layers; i++)
        if (!layers[i] || !k_caches[i] || !v_caches[i]) return fail(W4_EINVAL, "null layer or cache %d", i);
    if (layers[0]->cfg.hidden != lm->cfg.hidden) return fail(W4_EINVAL, "layers and LM ends differ in hidden size");
    if (B < 1 || max_ctx < 0) return fail(W4_EINVAL, "B must be >= 1 and max_ctx >= 0");
    if (B > lm->cfg.max_batch) return fail(W4_ECAPACITY, "B %d > the LM ends' max_batch %d", B, lm->cfg.max_batch);
    int rc;
    if ((rc = model_check(layers, n_layers, B, max_ctx))) return rc;
    const size_t need = model_decode_workspace_size(layers, n_layers, lm, B, max_ctx);
    if (need == 0) return fail(W4_ECAPACITY, "B or max_ctx outside what the layers hold");
    if (!ws || ws_bytes < need) return fail(W4_EWORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
    const size_t act = model_act_bytes(B, lm->cfg.hidden);
    float* x = (float*)ws;
    float* y = (float*)((char*)ws + act);
    void* rest = (char*)ws + 2 * act;
    const size_t sbytes = ws_bytes - 2 * act;
    if ((rc = lm_embed(lm, tokens, B, x, stream))) return rc;
    if ((rc = stack_decode(layers, n_layers, x, pos, ctx_lens, max_ctx, nullptr, B, k_caches, v_caches, y, rest,
                           sbytes, stream)))
        return rc;
    if ((rc = lm_head(lm, y, B, logits, next_tokens, rest, sbytes, stream))) return rc;
    // a raised error flag (the LM's or any layer's) turns the picks into -1,
    // so a loop that stays on the device sees the failure in its tokens
    std::vector<const int*> flags{(const int*)lm->err.p};
    for (int i = 0; i < n_layers; i++) flags.push_back(layers[i]->err);
    if (launch_pick_guard(flags.data(), (int)flags.size(), next_tokens, B, (hipStream_t)stream))
        return fail(W4_EHIP, "kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
    return W4_OK;
}

}  // extern "C"
