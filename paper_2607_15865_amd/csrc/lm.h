// Launchers of the model-end kernels (lm.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

// Model ends (lm.hip): embedding gather table[tokens[b]] -> fp32 out [B][H]
// (H % 4 == 0; an id outside [0, V) gives a zero row and sets *err), and the
// greedy pick next[b] = argmax_v logits[b][v] (lowest index among equal
// maxima; V % 4 == 0) with argmax_blocks(V) (value, index) pairs per row of
// scratch in pv / pi.
int launch_embed(const uint16_t* table, const int32_t* tokens, int V, int H, int B, float* out, int* err,
                 hipStream_t stream);
int argmax_blocks(int V);
int launch_argmax(const float* logits, int B, int V, float* pv, int* pi, int32_t* next, hipStream_t stream);
// After a pick: next[0..B) = -1 if any of the n error words flags[i] (device
// ints) is non-zero.
int launch_pick_guard(const int* const* flags, int n, int32_t* next, int B, hipStream_t stream);
