// Transformer problems (decoder-only, pre-LayerNorm, RoPE) with per-token loss
// weights from a meta-model: layout, workspace sizes and the three entry
// points, called by the C ABI front end.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

#include "mfmg.h"

namespace mfmg {

// Returns nullptr if desc describes a supported transformer problem, else a message.
const char* tf_validate(const mfmg_problem_desc& d);
long tf_n_theta(const mfmg_problem_desc& d);
long tf_n_eta(const mfmg_problem_desc& d);
size_t tf_meta_ws(const mfmg_problem_desc& d, int T, size_t* static_bytes, size_t* dynamic_bytes);
size_t tf_step_ws(const mfmg_problem_desc& d);

hipError_t tf_run_meta(const mfmg_problem_desc& d, const float* theta0, const float* eta,
                       const mfmg_batch* batches, int T, const mfmg_batch* val, float* d_eta,
                       float* val_loss, char* ws, hipStream_t s);
hipError_t tf_run_inner(const mfmg_problem_desc& d, const float* theta, const float* eta,
                        const mfmg_batch* b, float* theta_next, float* grad_out, float* loss_out,
                        char* ws, hipStream_t s);
hipError_t tf_run_hvp(const mfmg_problem_desc& d, const float* theta, const float* eta,
                      const mfmg_batch* b, const float* v, float* grad_out, float* hvp_out,
                      float* mvp_out, char* ws, hipStream_t s);

}  // namespace mfmg
