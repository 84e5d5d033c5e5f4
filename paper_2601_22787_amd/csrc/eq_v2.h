// Version-2 containers (tile-ordered chunks, phrase alphabet): the entry
// points of eq.h hand a version-2 layer to these (eq_decode2.hip).
#pragma once
#include "eq.h"

namespace eq_detail {
int v2_prepare(const eq_layer *L, hipStream_t s);
int v2_decode_codes(const eq_layer *L, uint8_t *codes, hipStream_t s);
int v2_decode_bf16(const eq_layer *L, uint16_t *w, hipStream_t s);
size_t v2_gemv_workspace_bytes(const eq_layer *L, uint32_t B);
int v2_decode_gemv(const eq_layer *L, const uint16_t *x, uint32_t B, const uint16_t *bias,
                   float *y, void *ws, size_t ws_bytes, hipStream_t s);
bool v2_layer_ok(const eq_layer *L);
// Layers that one version-2 launch can decode together: 2..8 valid version-2
// layers with one tile height and one input width.
bool v2_joint_ok(const eq_layer *const *L, uint32_t n);
// Fused GEMV of n such layers reading the same x; ws[i] is layer i's
// workspace (v2_gemv_workspace_bytes(L[i], B)).
int v2_decode_gemv_multi(const eq_layer *const *L, uint32_t n, const uint16_t *x, uint32_t B,
                         const uint16_t *const *bias, float *const *y, void *const *ws,
                         hipStream_t s);
// Layers that one version-2 launch can decode to codes or BF16 together:
// 2..8 valid version-2 layers (of any tile heights).
bool v2_joint_out_ok(const eq_layer *const *L, uint32_t n);
// Codes or BF16 of n such layers, layer i to codes[i] / w[i], in one launch.
int v2_decode_codes_multi(const eq_layer *const *L, uint8_t *const *codes, uint32_t n,
                          hipStream_t s);
int v2_decode_bf16_multi(const eq_layer *const *L, uint16_t *const *w, uint32_t n,
                         hipStream_t s);
}  // namespace eq_detail
