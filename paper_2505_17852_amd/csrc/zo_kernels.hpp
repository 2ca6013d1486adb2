// Launchers of the HIP kernels (host side). Every launcher only enqueues on
// `stream`; argument checking happens in the C ABI layer before these run.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "zo_common.hpp"

namespace zo {

// k_rng.hip
hipError_t launch_debug_probe(int kind, uint64_t seed, uint32_t i, uint64_t j0, uint64_t n,
                              float* out, hipStream_t s);
hipError_t launch_debug_gauss_pairs(const uint32_t* words, uint64_t n_pairs, float* out,
                                    hipStream_t s);
hipError_t launch_init(int wdtype, void* theta, uint64_t P, uint64_t seed, float scale,
                       hipStream_t s);
// lm_stride 1: Lm holds one loss per probe (central differences); 0: one
// loss for all probes (forward differences: the clean pass, with eps halved
// by the caller so that the coefficient divides by eps).
// bits: the sign words of the probes (zo_update_cached; sign probes only), or
// nullptr to regenerate them.
hipError_t launch_update(int wdtype, int kind, void* theta, uint64_t P, uint64_t seed, float eps,
                         float lr, int32_t N, uint32_t i0, const float* Lp, const float* Lm,
                         int32_t* skipped, hipStream_t s, int lm_stride = 1, const uint32_t* bits = nullptr);
// The sign words of probes i0 .. i0+N-1 into bits (layout: bit_words).
hipError_t launch_bits_fill(uint32_t* bits, uint64_t P, uint64_t seed, uint32_t i0, int32_t N, hipStream_t s);

// k_forward.hip: one call of the perturbed forward passes.
struct ForwardArgs {
  zo_config cfg;
  Layout lay;
  Rows rows;
  WsPlan ws;
  const void* theta;
  uint64_t seed;
  float eps;
  uint32_t i0;
  const int32_t* tokens;
  const uint8_t* mask;
  int32_t C;
  float* Lplus;
  float* Lminus;
  char* work;
  bool split;       // two-stream products: A.W and A.(s eps z) as separate MFMA streams into one
                    // accumulator (bf16 weights: eps below the fused form's floor; fp32: measurement)
  void* zc;         // probe cache inside work, or nullptr (probes regenerated in every tile)
  uint32_t* bits;   // sign-probe cache inside work (bf16 weights, sign probes), or nullptr
  void* w16;        // bf16 weights: fp16 copy of the product matrices inside work (ZCacheMap layout)
  ZCacheMap zmap;
};
hipError_t launch_forward(const ForwardArgs& a, hipStream_t s);

// k_forward_bf16.hip: the bf16 path's per-timestep kernels.
hipError_t launch_embed_bf16(const ForwardArgs& a, int t, void* x0, hipStream_t st);
hipError_t launch_gate_bf16(const ForwardArgs& a, int l, const void* x, const void* hprev, void* hout,
                            float* cst, const float* zb, hipStream_t st);
hipError_t launch_head_bf16(const ForwardArgs& a, const void* hist, int t0, int Tc, const float* zbo,
                            float* pmax, float* psum, float* ptgt, hipStream_t st);

}  // namespace zo
