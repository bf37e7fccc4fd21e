// launch.h -- host-side launchers of the libmxattn kernels (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mxattn {

// Shared-scale rule of the MXFP4 quantizer.
// kRuleQmax is the ceil rule of a general boundary q (Boundary in
// device_common.h), a run-time argument of the quantizers.
enum Rule { kRuleOcp = 0, kRuleUos = 1, kRuleQmax = 2 };

// Query rows per workgroup of the fused attention kernel, and its KV tile
// B_c: the running maximum is updated once per kKvTile keys.
constexpr int kQueryTile = 128;
constexpr int kKvTile = 128;

hipError_t launch_quantize_headdim(const void* x, uint8_t* codes, uint8_t* scales, int64_t rows,
                                   int rule, hipStream_t stream, double qmax = 0.0);

// Q/K of the rotated mode: rows multiplied by R_H = H/sqrt(128) first.
hipError_t launch_quantize_headdim_rotated(const void* x, uint8_t* codes, uint8_t* scales, int64_t rows,
                                           int rule, hipStream_t stream);

hipError_t launch_quantize_tokens(const void* x, uint8_t* codes, uint8_t* scales, int64_t BH,
                                  int64_t N, int rule, hipStream_t stream, double qmax = 0.0);

// Per-head squared-error sweep over boundaries (qmax.hip).  The histogram
// pass writes partial sums to a workspace of qmax_sse_workspace_bytes(...)
// bytes; the reduction turns them into sse[BH, nq] (fp64).
constexpr int kMaxBoundaries = 64;
int64_t qmax_sse_workspace_bytes(int axis, int64_t BH, int64_t N);
hipError_t launch_qmax_sse(const void* x, int axis, const double* qs, int nq, double* sse,
                           void* workspace, int64_t BH, int64_t N, hipStream_t stream);

struct AttnArgs {
    const uint8_t* qc;  // [BH, Nq, 64]
    const uint8_t* qs;  // [BH, Nq, 4]
    const uint16_t* qraw;  // bf16 Q [BH, Nq, 128] if the kernel quantizes Q itself, else null
    const uint8_t* kc;  // [BH, N, 64]
    const uint8_t* ks;  // [BH, N, 4]
    const uint8_t* vc;  // [BH, 128, nb * 16]
    const uint8_t* vs;  // [BH, 128, nb]
    const uint8_t* sc;  // [BH, ntiles, 1024]: K^ and V^ scales in MFMA operand order
    uint16_t* out;      // [BH, Nq, 128] bf16
    int N;              // keys / values per head
    int Nq;             // queries per head (Q^ codes/scales and out are [BH, Nq, ...])
    int nb;
    int qtiles;
    int total_tiles;    // workgroups that do work
    int per_xcd;
    int nchunks;        // resident kernel: workgroups per (batch, head)
};

// Largest key (and value) length of the fused attention kernel: one head's
// K^ codes (64 B per key) and V^ codes (128 channels x 16 B per 32 keys) are
// addressed through buffer resources with 32-bit byte offsets, which stay
// below 2^31 up to this length.
constexpr int64_t kMaxKeys = (int64_t)1 << 24;

// Keys up to which the whole of K^ and V^ of a head stays in LDS for the
// workgroup's lifetime (launch_attention then runs the resident kernel).
constexpr int kResidentKeys = 512;

// Scales of K^ and V^ in the attention kernel's operand order (AttnArgs::sc);
// out holds tile_scales_bytes(BH, N) bytes.
inline int64_t tile_scales_bytes(int64_t BH, int64_t N) { return BH * ((N + 127) / 128) * 1024; }
hipError_t launch_tile_scales(const uint8_t* ks, const uint8_t* vs, uint8_t* out, int64_t BH, int64_t N,
                              hipStream_t stream);

// Row-sum diagnostics (rowsum.hip).  Attention rows [row0, row0 + rows) of
// every head: either p [BH, rows, ld] fp32 stored, or their quantization
// statistics written to stats [BH, Nq, 8] (fp64).
enum RowsOut { kRowsStoreP = 0, kRowsDiagUos = 1, kRowsDiagOcp = 2 };
struct SoftmaxRowsArgs {
    const uint16_t* q;  // [BH, Nq, 128] bf16
    const uint16_t* k;  // [BH, Nkv, 128] bf16
    float* p;           // [BH, rows, ld] (kRowsStoreP)
    int Nq, Nkv, row0, rows, ld;
    float gamma;        // pre-scale (diagnostics)
    double g;           // fp64(1 / gamma)
    double* stats;      // [BH, Nq, 8] (diagnostics)
    int qtiles;         // set by the launcher
    float c;            // set by the launcher: log2(e) / sqrt(128)
};
hipError_t launch_attn_rows(const SoftmaxRowsArgs& a, int64_t BH, int out, hipStream_t stream);

// Diagnostics of rows of p [n_rows, ld] (first N entries), written to
// stats[((r / rows_per_head) * out_rows_per_head + out_row0 + r % rows_per_head) * 8 + i].
struct RowsumDiagArgs {
    const float* p;
    int64_t N, ld;
    float gamma;  // pre-scale
    double g;     // fp64(1 / gamma)
    double* stats;
    int64_t rows_per_head, out_rows_per_head, out_row0;
};
hipError_t launch_rowsum_diag(const RowsumDiagArgs& a, int64_t n_rows, int rule, hipStream_t stream);

// mode: 0 OCP + direct, 1 UOS + direct, 2 UOS + PNQ
hipError_t launch_attention(const AttnArgs& a, int mode, hipStream_t stream);

}  // namespace mxattn
