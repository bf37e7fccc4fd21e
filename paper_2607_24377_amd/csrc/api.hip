// api.hip -- the extern "C" entry points of libmxattn (see include/mxattn.h).
//
// Argument validation happens before any HIP call, so every error path is
// free of device work.  The only global state is the library's own
// stream-ordered workspace pool per device (created once, see
// workspace_alloc).
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "../../include/mxattn.h"
#include "launch.h"

namespace {

thread_local char g_last_error[256] = "";

void set_error(const char* what, hipError_t e) {
    std::snprintf(g_last_error, sizeof g_last_error, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// Whether the byte ranges [a, a + na) and [b, b + nb) share a byte.
bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + nb && y < x + na;
}

bool valid_mode(int mode) { return mode >= MXATTN_OCP_VANILLA && mode <= MXATTN_UOS_PNQ_ROT; }

// The attention kernel's mode: the rotated mode differs only in how Q and K
// were quantized.
int kernel_mode(int mode) { return mode == MXATTN_UOS_PNQ_ROT ? MXATTN_UOS_PNQ : mode; }

// Shape limits of the kernels: 32-bit token indices, 64-bit byte offsets, and
// at most 2^35 elements per tensor (64 GiB of bf16), which keeps every grid
// below 2^31 workgroups.
int check_shape(int64_t B, int64_t H, int64_t N, int64_t d) {
    if (B < 1 || H < 1 || N < 1 || d < 1) return MXATTN_ERR_SHAPE;
    if (B > (1 << 20) || H > (1 << 20) || N > (1 << 28)) return MXATTN_ERR_SHAPE;
    if (B * H > (int64_t)1 << 24) return MXATTN_ERR_SHAPE;
    if (B * H * N * 128 > (int64_t)1 << 35) return MXATTN_ERR_SHAPE;
    if (d != 128) return MXATTN_ERR_UNSUPPORTED;
    return MXATTN_OK;
}

int rule_of(int mode) { return mode == MXATTN_OCP_VANILLA ? mxattn::kRuleOcp : mxattn::kRuleUos; }

constexpr int kMaxDevices = 64;

// Workspace memory comes from a stream-ordered pool that belongs to the
// library, one per device, created on first use.  Its release threshold has
// no limit, so the forward's workspace is recycled between calls instead of
// being returned to the driver at every synchronization; the device's
// default pool, which other libraries share, keeps its attributes.
// mxattn_release_workspace() hands the cached memory back.  If the pool
// cannot be created, workspace comes from the default pool (unchanged).
struct PoolSlot {
    std::once_flag once;
    std::atomic<hipMemPool_t> pool{nullptr};
};
PoolSlot g_pools[kMaxDevices];

hipMemPool_t private_pool(int dev) {
    if (dev < 0 || dev >= kMaxDevices) return nullptr;
    PoolSlot& slot = g_pools[dev];
    std::call_once(slot.once, [dev, &slot] {
        hipMemPoolProps props{};
        props.allocType = hipMemAllocationTypePinned;
        props.handleTypes = hipMemHandleTypeNone;
        props.location.type = hipMemLocationTypeDevice;
        props.location.id = dev;
        hipMemPool_t pool = nullptr;
        if (hipMemPoolCreate(&pool, &props) != hipSuccess || !pool) {
            (void)hipGetLastError();
            return;
        }
        uint64_t threshold = UINT64_MAX;
        if (hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &threshold) != hipSuccess) {
            (void)hipGetLastError();
            (void)hipMemPoolDestroy(pool);
            return;
        }
        slot.pool.store(pool);
    });
    return slot.pool.load();
}

hipError_t workspace_alloc(void** p, size_t bytes, hipStream_t s) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
    if (hipMemPool_t pool = private_pool(dev)) return hipMallocFromPoolAsync(p, bytes, pool, s);
    return hipMallocAsync(p, bytes, s);
}

}  // namespace

extern "C" {

int mxattn_version(void) { return 101; }

int mxattn_release_workspace(void) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        set_error("hipGetDevice", e);
        return MXATTN_ERR_HIP;
    }
    if (dev < 0 || dev >= kMaxDevices) return MXATTN_OK;
    hipMemPool_t pool = g_pools[dev].pool.load();
    if (!pool) return MXATTN_OK;  // no workspace was ever taken on this device
    e = hipMemPoolTrimTo(pool, 0);
    if (e != hipSuccess) {
        set_error("hipMemPoolTrimTo", e);
        return MXATTN_ERR_HIP;
    }
    return MXATTN_OK;
}

int mxattn_kv_tile(void) { return mxattn::kKvTile; }

int mxattn_query_tile(void) { return mxattn::kQueryTile; }

const char* mxattn_status_string(int s) {
    switch (s) {
        case MXATTN_OK: return "ok";
        case MXATTN_ERR_NULL: return "null pointer argument";
        case MXATTN_ERR_SHAPE: return "invalid shape (B, H, N must be >= 1 and within limits)";
        case MXATTN_ERR_ALIGN: return "misaligned pointer (tensors need 16-byte alignment)";
        case MXATTN_ERR_MODE: return "invalid mode (0 ocp_vanilla, 1 uos, 2 uos_pnq, 3 uos_pnq_rot)";
        case MXATTN_ERR_AXIS: return "invalid block_axis (2 = tokens, 3 = head dim)";
        case MXATTN_ERR_UNSUPPORTED: return "unsupported head dimension (d must be 128)";
        case MXATTN_ERR_OOM: return "workspace allocation failed";
        case MXATTN_ERR_HIP: return "HIP runtime error";
        case MXATTN_ERR_SCRATCH: return "problem too large for the static scratch of the no-allocation entry point (needs B*H*ceil(Nkv/128) <= 32768)";
        case MXATTN_ERR_BOUNDARY: return "invalid scale boundary (need 4 <= q <= 8 and 1 <= nq <= 64) or pre-scale (need 0 < gamma < 3e38)";
        default: return "unknown status";
    }
}

const char* mxattn_last_error(void) { return g_last_error; }

size_t mxattn_codes_bytes(int block_axis, int64_t B, int64_t H, int64_t N, int64_t d) {
    if (check_shape(B, H, N, d) != MXATTN_OK) return 0;
    if (block_axis == MXATTN_AXIS_HEAD_DIM) return (size_t)(B * H * N * (d / 2));
    if (block_axis == MXATTN_AXIS_TOKENS) return (size_t)(B * H * d * ((N + 31) / 32) * 16);
    return 0;
}

size_t mxattn_scales_bytes(int block_axis, int64_t B, int64_t H, int64_t N, int64_t d) {
    if (check_shape(B, H, N, d) != MXATTN_OK) return 0;
    if (block_axis == MXATTN_AXIS_HEAD_DIM) return (size_t)(B * H * N * (d / 32));
    if (block_axis == MXATTN_AXIS_TOKENS) return (size_t)(B * H * d * ((N + 31) / 32));
    return 0;
}

int mxattn_quantize(const void* x, uint8_t* codes, uint8_t* scales, int block_axis, int mode,
                    int64_t B, int64_t H, int64_t N, int64_t d, void* stream) {
    if (!x || !codes || !scales) return MXATTN_ERR_NULL;
    if (block_axis != MXATTN_AXIS_HEAD_DIM && block_axis != MXATTN_AXIS_TOKENS) return MXATTN_ERR_AXIS;
    if (!valid_mode(mode)) return MXATTN_ERR_MODE;
    if (int st = check_shape(B, H, N, d)) return st;
    if (!aligned(x, 16) || !aligned(codes, 16)) return MXATTN_ERR_ALIGN;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t e;
    if (block_axis == MXATTN_AXIS_HEAD_DIM && mode == MXATTN_UOS_PNQ_ROT)
        e = mxattn::launch_quantize_headdim_rotated(x, codes, scales, B * H * N, rule_of(mode), s);
    else if (block_axis == MXATTN_AXIS_HEAD_DIM)
        e = mxattn::launch_quantize_headdim(x, codes, scales, B * H * N, rule_of(mode), s);
    else
        e = mxattn::launch_quantize_tokens(x, codes, scales, B * H, N, rule_of(mode), s);
    if (e != hipSuccess) {
        set_error("quantize launch", e);
        return MXATTN_ERR_HIP;
    }
    return MXATTN_OK;
}

int mxattn_quantize_qmax(const void* x, uint8_t* codes, uint8_t* scales, int block_axis, double qmax,
                         int64_t B, int64_t H, int64_t N, int64_t d, void* stream) {
    if (!x || !codes || !scales) return MXATTN_ERR_NULL;
    if (block_axis != MXATTN_AXIS_HEAD_DIM && block_axis != MXATTN_AXIS_TOKENS) return MXATTN_ERR_AXIS;
    if (!(qmax >= 4.0 && qmax <= 8.0)) return MXATTN_ERR_BOUNDARY;
    if (int st = check_shape(B, H, N, d)) return st;
    if (!aligned(x, 16) || !aligned(codes, 16)) return MXATTN_ERR_ALIGN;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t e = block_axis == MXATTN_AXIS_HEAD_DIM
                       ? mxattn::launch_quantize_headdim(x, codes, scales, B * H * N, mxattn::kRuleQmax, s, qmax)
                       : mxattn::launch_quantize_tokens(x, codes, scales, B * H, N, mxattn::kRuleQmax, s, qmax);
    if (e != hipSuccess) {
        set_error("quantize launch", e);
        return MXATTN_ERR_HIP;
    }
    return MXATTN_OK;
}

int mxattn_qmax_sse(const void* x, int block_axis, const double* qs, int nq, double* sse, int64_t B,
                    int64_t H, int64_t N, int64_t d, void* stream) {
    if (!x || !qs || !sse) return MXATTN_ERR_NULL;
    if (block_axis != MXATTN_AXIS_HEAD_DIM && block_axis != MXATTN_AXIS_TOKENS) return MXATTN_ERR_AXIS;
    if (nq < 1 || nq > MXATTN_MAX_BOUNDARIES) return MXATTN_ERR_BOUNDARY;
    for (int j = 0; j < nq; j++)
        if (!(qs[j] >= 4.0 && qs[j] <= 8.0)) return MXATTN_ERR_BOUNDARY;
    if (int st = check_shape(B, H, N, d)) return st;
    if (!aligned(x, 16) || !aligned(sse, 8)) return MXATTN_ERR_ALIGN;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    void* ws = nullptr;
    hipError_t e = workspace_alloc(&ws, (size_t)mxattn::qmax_sse_workspace_bytes(block_axis, B * H, N), s);
    if (e != hipSuccess || !ws) {
        set_error("workspace allocation", e);
        return MXATTN_ERR_OOM;
    }
    int st = MXATTN_OK;
    e = mxattn::launch_qmax_sse(x, block_axis, qs, nq, sse, ws, B * H, N, s);
    if (e != hipSuccess) {
        set_error("sse sweep launch", e);
        st = MXATTN_ERR_HIP;
    }
    e = hipFreeAsync(ws, s);
    if (st == MXATTN_OK && e != hipSuccess) {
        set_error("hipFreeAsync", e);
        st = MXATTN_ERR_HIP;
    }
    return st;
}

int mxattn_softmax_rows(const void* q, const void* k, float* p, int64_t B, int64_t H, int64_t Nq,
                        int64_t Nkv, int64_t d, int64_t row0, int64_t rows, int64_t ld, void* stream) {
    if (!q || !k || !p) return MXATTN_ERR_NULL;
    if (int st = check_shape(B, H, Nq, d)) return st;
    if (int st = check_shape(B, H, Nkv, d)) return st;
    if (row0 < 0 || rows < 1 || row0 + rows > Nq || ld < Nkv || ld % 4 != 0 || ld > (1 << 28))
        return MXATTN_ERR_SHAPE;
    const int64_t qtiles = (rows + 127) / 128;
    if (B * H * qtiles > ((int64_t)1 << 31) - 1) return MXATTN_ERR_SHAPE;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(p, 16)) return MXATTN_ERR_ALIGN;
    mxattn::SoftmaxRowsArgs a{};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.p = p;
    a.Nq = (int)Nq;
    a.Nkv = (int)Nkv;
    a.row0 = (int)row0;
    a.rows = (int)rows;
    a.ld = (int)ld;
    hipError_t e = mxattn::launch_attn_rows(a, B * H, mxattn::kRowsStoreP, reinterpret_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        set_error("softmax rows launch", e);
        return MXATTN_ERR_HIP;
    }
    return MXATTN_OK;
}

static bool valid_gamma(float gamma) { return gamma > 0.0f && gamma < 3.0e38f; }

int mxattn_rowsum_diag(const float* p, int64_t rows, int64_t N, int64_t ld, int mode, float gamma,
                       double* stats, void* stream) {
    if (!p || !stats) return MXATTN_ERR_NULL;
    if (!valid_mode(mode)) return MXATTN_ERR_MODE;
    if (rows < 1 || rows > ((int64_t)1 << 31) - 1 || N < 1 || N > (1 << 28) || ld < N || ld % 4 != 0)
        return MXATTN_ERR_SHAPE;
    if (!valid_gamma(gamma)) return MXATTN_ERR_BOUNDARY;
    if (!aligned(p, 16) || !aligned(stats, 8)) return MXATTN_ERR_ALIGN;
    mxattn::RowsumDiagArgs a{};
    a.p = p;
    a.N = N;
    a.ld = ld;
    a.gamma = gamma;
    a.g = 1.0 / (double)gamma;
    a.stats = stats;
    a.rows_per_head = rows;
    a.out_rows_per_head = rows;
    a.out_row0 = 0;
    hipError_t e = mxattn::launch_rowsum_diag(a, rows, rule_of(mode), reinterpret_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        set_error("row-sum diagnostic launch", e);
        return MXATTN_ERR_HIP;
    }
    return MXATTN_OK;
}

int mxattn_attention_rowsum_diag(const void* q, const void* k, int64_t B, int64_t H, int64_t Nq,
                                 int64_t Nkv, int64_t d, int mode, float gamma, double* stats,
                                 void* stream) {
    if (!q || !k || !stats) return MXATTN_ERR_NULL;
    if (!valid_mode(mode)) return MXATTN_ERR_MODE;
    if (int st = check_shape(B, H, Nq, d)) return st;
    if (int st = check_shape(B, H, Nkv, d)) return st;
    if (!valid_gamma(gamma)) return MXATTN_ERR_BOUNDARY;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(stats, 8)) return MXATTN_ERR_ALIGN;
    if (B * H * ((Nq + 127) / 128) > ((int64_t)1 << 31) - 1) return MXATTN_ERR_SHAPE;
    mxattn::SoftmaxRowsArgs a{};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.Nq = (int)Nq;
    a.Nkv = (int)Nkv;
    a.row0 = 0;
    a.rows = (int)Nq;
    a.gamma = gamma;
    a.g = 1.0 / (double)gamma;
    a.stats = stats;
    const int out = rule_of(mode) == mxattn::kRuleUos ? mxattn::kRowsDiagUos : mxattn::kRowsDiagOcp;
    hipError_t e = mxattn::launch_attn_rows(a, B * H, out, reinterpret_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        set_error("row-sum diagnostic launch", e);
        return MXATTN_ERR_HIP;
    }
    return MXATTN_OK;
}

// Limits of the fused attention kernel beyond check_shape: the key length
// (32-bit byte offsets within one head's K^/V^) and the workgroup count.
int check_attention_shape(int64_t B, int64_t H, int64_t Nq, int64_t Nkv) {
    if (Nkv > mxattn::kMaxKeys) return MXATTN_ERR_SHAPE;
    if (B * H * ((Nq + mxattn::kQueryTile - 1) / mxattn::kQueryTile) > (int64_t)1 << 30) return MXATTN_ERR_SHAPE;
    return MXATTN_OK;
}

// Rearranges the K^/V^ scales into sc (mxattn::tile_scales_bytes(B*H, Nkv)
// bytes of workspace), then runs the fused attention kernel: on Q^ = (qc, qs),
// or, when qraw is not null, on the bf16 Q that the kernel quantizes itself
// (qc and qs are then unused).
static int launch_attend(const void* qraw, const uint8_t* qc, const uint8_t* qs, const uint8_t* kc,
                         const uint8_t* ks, const uint8_t* vc, const uint8_t* vs, uint8_t* sc,
                         void* out, int64_t B, int64_t H, int64_t Nq, int64_t Nkv, int mode,
                         hipStream_t s) {
    hipError_t e = mxattn::launch_tile_scales(ks, vs, sc, B * H, Nkv, s);
    if (e != hipSuccess) {
        set_error("scale layout launch", e);
        return MXATTN_ERR_HIP;
    }
    mxattn::AttnArgs a;
    a.qc = qc;
    a.qs = qs;
    a.qraw = static_cast<const uint16_t*>(qraw);
    a.kc = kc;
    a.ks = ks;
    a.vc = vc;
    a.vs = vs;
    a.sc = sc;
    a.out = static_cast<uint16_t*>(out);
    a.N = (int)Nkv;
    a.Nq = (int)Nq;
    a.nb = (int)((Nkv + 31) / 32);
    a.qtiles = (int)((Nq + mxattn::kQueryTile - 1) / mxattn::kQueryTile);
    // one query tile per workgroup; with K^/V^ resident in LDS, chunks of at
    // most 16 query tiles, as many as fill whole rounds of the 512 workgroups
    // resident at once (two per CU), split evenly by the kernel
    int64_t nchunks = a.qtiles;
    if (Nkv <= mxattn::kResidentKeys) {
        const int64_t slots = 512, bh = B * H;
        const int64_t min_chunks = (a.qtiles + 15) / 16;
        const int64_t rounds = (bh * min_chunks + slots - 1) / slots;
        const int64_t k = rounds * slots / bh;
        nchunks = k < min_chunks ? min_chunks : (k > a.qtiles ? a.qtiles : k);
    }
    a.nchunks = (int)nchunks;
    const int64_t total = B * H * a.nchunks;
    a.total_tiles = (int)total;
    a.per_xcd = (int)((total + 7) / 8);
    e = mxattn::launch_attention(a, kernel_mode(mode), s);
    if (e != hipSuccess) {
        set_error("attention launch", e);
        return MXATTN_ERR_HIP;
    }
    return MXATTN_OK;
}

// Whether `out` ([B, H, Nq, d] bf16) shares memory with any quantized operand.
static bool attend_out_aliases(const uint8_t* qc, const uint8_t* qs, const uint8_t* kc, const uint8_t* ks,
                               const uint8_t* vc, const uint8_t* vs, const void* out, int64_t B, int64_t H,
                               int64_t Nq, int64_t Nkv, int64_t d) {
    const size_t ob = (size_t)(B * H * Nq * d * 2);
    return overlaps(out, ob, qc, mxattn_codes_bytes(MXATTN_AXIS_HEAD_DIM, B, H, Nq, d)) ||
           overlaps(out, ob, qs, mxattn_scales_bytes(MXATTN_AXIS_HEAD_DIM, B, H, Nq, d)) ||
           overlaps(out, ob, kc, mxattn_codes_bytes(MXATTN_AXIS_HEAD_DIM, B, H, Nkv, d)) ||
           overlaps(out, ob, ks, mxattn_scales_bytes(MXATTN_AXIS_HEAD_DIM, B, H, Nkv, d)) ||
           overlaps(out, ob, vc, mxattn_codes_bytes(MXATTN_AXIS_TOKENS, B, H, Nkv, d)) ||
           overlaps(out, ob, vs, mxattn_scales_bytes(MXATTN_AXIS_TOKENS, B, H, Nkv, d));
}

// Argument checks of the attention calls on quantized operands.
static int check_attend_args(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                             const uint8_t* k_scales, const uint8_t* v_codes, const uint8_t* v_scales,
                             const void* out, int64_t B, int64_t H, int64_t Nq, int64_t Nkv, int64_t d,
                             int mode) {
    if (!q_codes || !q_scales || !k_codes || !k_scales || !v_codes || !v_scales || !out)
        return MXATTN_ERR_NULL;
    if (!valid_mode(mode)) return MXATTN_ERR_MODE;
    if (int st = check_shape(B, H, Nq, d)) return st;
    if (int st = check_shape(B, H, Nkv, d)) return st;
    if (int st = check_attention_shape(B, H, Nq, Nkv)) return st;
    if (!aligned(q_codes, 16) || !aligned(k_codes, 16) || !aligned(v_codes, 16) ||
        !aligned(out, 16) || !aligned(k_scales, 4))
        return MXATTN_ERR_ALIGN;
    if (attend_out_aliases(q_codes, q_scales, k_codes, k_scales, v_codes, v_scales, out, B, H, Nq, Nkv, d))
        return MXATTN_ERR_SHAPE;
    return MXATTN_OK;
}

int mxattn_cross_attend(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                        const uint8_t* k_scales, const uint8_t* v_codes, const uint8_t* v_scales,
                        void* out, int64_t B, int64_t H, int64_t Nq, int64_t Nkv, int64_t d, int mode,
                        void* stream) {
    if (int st = check_attend_args(q_codes, q_scales, k_codes, k_scales, v_codes, v_scales, out, B, H, Nq, Nkv,
                                   d, mode))
        return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    void* ws = nullptr;
    hipError_t e = workspace_alloc(&ws, (size_t)mxattn::tile_scales_bytes(B * H, Nkv), s);
    if (e != hipSuccess || !ws) {
        set_error("workspace allocation", e);
        return MXATTN_ERR_OOM;
    }
    int st = launch_attend(nullptr, q_codes, q_scales, k_codes, k_scales, v_codes, v_scales,
                           static_cast<uint8_t*>(ws), out, B, H, Nq, Nkv, mode, s);
    e = hipFreeAsync(ws, s);
    if (st == MXATTN_OK && e != hipSuccess) {
        set_error("hipFreeAsync", e);
        st = MXATTN_ERR_HIP;
    }
    return st;
}

// ---- the entry point that allocates nothing
//
// mxattn_cross_attend_noalloc keeps its one buffer beyond the inputs and the
// output, the K^/V^ scales rearranged into MFMA operand order (1 KiB per
// (batch, head) and 128-key tile), in this static device array instead of
// allocated workspace.  Each device the library runs on holds its own copy
// until the process ends.  On the host, `scratch` is only a stand-in symbol,
// never a device address: the device address comes from hipGetSymbolAddress,
// taken once per device with that device current, and only that address is
// passed to kernels.  Every call on a device shares the device's array, so
// calls that overlap in time on one device race.
static __device__ __align__(256) uint8_t scratch[MXATTN_NOALLOC_SCRATCH_BYTES];

struct ScratchSlot {
    std::once_flag once;
    hipError_t err = hipSuccess;
    void* ptr = nullptr;
};
ScratchSlot g_scratch[kMaxDevices];

// The current device's address of `scratch` (looked up on the first call on
// that device).
static int scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        set_error("hipGetDevice", e);
        return MXATTN_ERR_HIP;
    }
    if (dev < 0 || dev >= kMaxDevices) {
        set_error("device index beyond the library's limit", hipErrorInvalidDevice);
        return MXATTN_ERR_HIP;
    }
    ScratchSlot& slot = g_scratch[dev];
    std::call_once(slot.once, [&slot] {
        void* p = nullptr;
        slot.err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (slot.err == hipSuccess && p)
            slot.ptr = p;
        else
            (void)hipGetLastError();
    });
    if (slot.err != hipSuccess || !slot.ptr) {
        set_error("hipGetSymbolAddress(scratch)", slot.err != hipSuccess ? slot.err : hipErrorInvalidSymbol);
        return MXATTN_ERR_HIP;
    }
    *out = slot.ptr;
    return MXATTN_OK;
}

int mxattn_cross_attend_noalloc(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                                const uint8_t* k_scales, const uint8_t* v_codes, const uint8_t* v_scales,
                                void* out, int64_t B, int64_t H, int64_t Nq, int64_t Nkv, int64_t d,
                                int mode, void* stream) {
    if (int st = check_attend_args(q_codes, q_scales, k_codes, k_scales, v_codes, v_scales, out, B, H, Nq, Nkv,
                                   d, mode))
        return st;
    const int64_t need = mxattn::tile_scales_bytes(B * H, Nkv);
    if (need > (int64_t)MXATTN_NOALLOC_SCRATCH_BYTES) {
        std::snprintf(g_last_error, sizeof g_last_error,
                      "mxattn_cross_attend_noalloc: %lld bytes of scale scratch needed (B*H*ceil(Nkv/128) KiB), "
                      "the static buffer holds %lld",
                      (long long)need, (long long)MXATTN_NOALLOC_SCRATCH_BYTES);
        return MXATTN_ERR_SCRATCH;
    }
    void* sc = nullptr;
    if (int st = scratch_address(&sc)) return st;
    return launch_attend(nullptr, q_codes, q_scales, k_codes, k_scales, v_codes, v_scales, static_cast<uint8_t*>(sc),
                         out, B, H, Nq, Nkv, mode, reinterpret_cast<hipStream_t>(stream));
}

int mxattn_attend(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                  const uint8_t* k_scales, const uint8_t* v_codes, const uint8_t* v_scales,
                  void* out, int64_t B, int64_t H, int64_t N, int64_t d, int mode, void* stream) {
    return mxattn_cross_attend(q_codes, q_scales, k_codes, k_scales, v_codes, v_scales, out, B, H, N,
                               N, d, mode, stream);
}

int mxattn_cross_forward(const void* q, const void* k, const void* v, void* out, int64_t B,
                         int64_t H, int64_t Nq, int64_t Nkv, int64_t d, int mode, void* stream) {
    if (!q || !k || !v || !out) return MXATTN_ERR_NULL;
    if (!valid_mode(mode)) return MXATTN_ERR_MODE;
    if (int st = check_shape(B, H, Nq, d)) return st;
    if (int st = check_shape(B, H, Nkv, d)) return st;
    if (int st = check_attention_shape(B, H, Nq, Nkv)) return st;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16))
        return MXATTN_ERR_ALIGN;
    {
        const size_t ob = (size_t)(B * H * Nq * d * 2), kb = (size_t)(B * H * Nkv * d * 2);
        if (overlaps(out, ob, q, ob) || overlaps(out, ob, k, kb) || overlaps(out, ob, v, kb))
            return MXATTN_ERR_SHAPE;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);

    // Q is quantized in the attention kernel's prologue (bit-identical to the
    // head-dim quantizer), except for the rotated mode, whose Q is rotated
    // across all 128 channels first by its own quantizer
    const bool q_fused = mode != MXATTN_UOS_PNQ_ROT;
    const size_t q_codes = q_fused ? 0 : mxattn_codes_bytes(MXATTN_AXIS_HEAD_DIM, B, H, Nq, d);
    const size_t q_scales = q_fused ? 0 : mxattn_scales_bytes(MXATTN_AXIS_HEAD_DIM, B, H, Nq, d);
    const size_t k_codes = mxattn_codes_bytes(MXATTN_AXIS_HEAD_DIM, B, H, Nkv, d);
    const size_t k_scales = mxattn_scales_bytes(MXATTN_AXIS_HEAD_DIM, B, H, Nkv, d);
    const size_t v_codes = mxattn_codes_bytes(MXATTN_AXIS_TOKENS, B, H, Nkv, d);
    const size_t v_scales = mxattn_scales_bytes(MXATTN_AXIS_TOKENS, B, H, Nkv, d);
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t tiled = (size_t)mxattn::tile_scales_bytes(B * H, Nkv);
    const size_t total = up(q_codes) + up(k_codes) + up(v_codes) + up(q_scales) + up(k_scales) +
                         up(v_scales) + up(tiled);

    void* ws = nullptr;
    hipError_t e = workspace_alloc(&ws, total, s);
    if (e != hipSuccess || !ws) {
        set_error("workspace allocation", e);
        return MXATTN_ERR_OOM;
    }
    uint8_t* p = static_cast<uint8_t*>(ws);
    uint8_t* qc = p;
    p += up(q_codes);
    uint8_t* kc = p;
    p += up(k_codes);
    uint8_t* vc = p;
    p += up(v_codes);
    uint8_t* qs = p;
    p += up(q_scales);
    uint8_t* ks = p;
    p += up(k_scales);
    uint8_t* vs = p;
    p += up(v_scales);
    uint8_t* sc = p;

    const int rule = rule_of(mode);
    int st = MXATTN_OK;
    auto qk = [mode](const void* x, uint8_t* c, uint8_t* sc, int64_t rows, int rule, hipStream_t st) {
        return mode == MXATTN_UOS_PNQ_ROT ? mxattn::launch_quantize_headdim_rotated(x, c, sc, rows, rule, st)
                                          : mxattn::launch_quantize_headdim(x, c, sc, rows, rule, st);
    };
    if ((!q_fused && (e = qk(q, qc, qs, B * H * Nq, rule, s)) != hipSuccess) ||
        (e = qk(k, kc, ks, B * H * Nkv, rule, s)) != hipSuccess ||
        (e = mxattn::launch_quantize_tokens(v, vc, vs, B * H, Nkv, rule, s)) != hipSuccess) {
        set_error("quantize launch", e);
        st = MXATTN_ERR_HIP;
    } else {
        st = launch_attend(q_fused ? q : nullptr, qc, qs, kc, ks, vc, vs, sc, out, B, H, Nq, Nkv, mode, s);
    }
    e = hipFreeAsync(ws, s);
    if (st == MXATTN_OK && e != hipSuccess) {
        set_error("hipFreeAsync", e);
        st = MXATTN_ERR_HIP;
    }
    return st;
}

int mxattn_forward(const void* q, const void* k, const void* v, void* out, int64_t B, int64_t H,
                   int64_t N, int64_t d, int mode, void* stream) {
    return mxattn_cross_forward(q, k, v, out, B, H, N, N, d, mode, stream);
}

}  // extern "C"
