// Launch interfaces between the C ABI (abi.hip) and the kernels. Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dbl {

constexpr int kTile = 128;            // vocabulary tile of the two-level log-prob form
constexpr int kTilesPerChunk = 32;    // vocabulary tiles per workgroup in the V-streaming kernels
constexpr int kMaxR = 64;             // categories handled by one wavefront

struct HeadArgs {
  int64_t M, V;
  int d;
  bool dtype_bf16;
  const void* h;
  const void* w;
  float* tls;
  float* lmass;
  float* lse;
  int32_t* argmax;      // [M] or null: lowest-index argmax of each row's logits
  uint64_t* amax_keys;  // workspace [M] when argmax is requested
};

// The branch log-probabilities and block description shared by the sampler and verifier.
struct BlockArgs {
  int64_t B, K, R, V;
  int nT;
  const float* tls;
  const float* lmass;
  const float* lse;
  const float* prior;  // [B, R]
  float z_temp;
  uint64_t seed, step;
  int64_t seq_offset;
};

struct SampleArgs {
  BlockArgs blk;
  int32_t* z_out;
  int32_t* x_out;
};

struct VerifyArgs {
  BlockArgs blk;
  const int32_t* x;     // [B, K]
  const float* logp;    // [B, Kp, V]
  int64_t Kp;
  bool trajectory;      // expected-length mode: no accept test, no residual
  int32_t* n_accept;    // [B] (verify only)
  int32_t* next_token;  // [B] (verify only)
  float* beta;          // [B, K] or null
  float* al;            // [B] or null
  float* exp_len;       // [B] or null
  double* wpost;        // workspace [B, K, R]: posterior weights
  float* beta_part;     // workspace [B*K, nchunk]
  uint64_t* res_tiles;  // workspace [B, nT]
  uint64_t* p_tiles;    // workspace [B, nT]
};

// Greedy-branch mode: the branch tokens replace the branch log-probabilities (blk.tls, lmass and
// lse are unused).
struct GreedyArgs {
  BlockArgs blk;
  const int32_t* xhat;  // [B, K, R] branch tokens argmax_v q_k(v | z)
  int32_t* z_out;       // sample: [B]
  int32_t* x_out;       // sample: [B, K]
  const int32_t* x;     // verify: [B, K] draft or trajectory
  const float* logp;    // verify: [B, Kp, V]
  int64_t Kp;
  bool trajectory;
  int32_t* n_accept;
  int32_t* next_token;
  float* beta;
  float* al;
  float* exp_len;
  double* wpost;        // workspace [B, K, R]
  uint64_t* res_tiles;  // workspace [B, nT]
  uint64_t* p_tiles;    // workspace [B, nT]
};

// Training-objective forward along target trajectories.
struct ObjectiveArgs {
  BlockArgs blk;
  const int32_t* x;     // [B, K] target trajectory
  const float* logp;    // [B, K, V]
  float tau;
  float* log_r;         // [B, K] or null
  float* S;             // [B, K] or null
  int32_t* ell_tau;     // [B]
  float* J;             // [B]
  float* nll;           // [B]
};

// Category hidden expander (bf16): out[m, z*d + j] = h[m, j] + (W h[m])[z*d + j] + c[z*d + j].
struct ExpandArgs {
  int64_t M, R;
  int d;
  const void* h;   // [M, d]
  const void* W;   // [R*d, d]
  const void* c;   // [R*d]
  void* out;       // [M, R*d]
};

// Category-prior head (bf16 inputs, fp32 logits): ell[b, z] = U[z] . h_anchor[b] + e[z].
struct PriorHeadArgs {
  int64_t B;
  int R, d;
  const void* h_anchor;  // [B, d]
  const void* U;         // [R, d]
  const void* e;         // [R]
  float* ell;            // [B, R]
};

// Target sampling transform: rows of logits -> filtered log-probabilities.
// Rows of the target transform split over kFilterSegs workgroups keep up to kFilterSegCap
// candidates each in the workspace.
constexpr int kFilterSegs = 4;
constexpr int kFilterSegCap = 1024;

struct FilterArgs {
  int64_t N, V;
  const float* logits;  // [N, V]
  float temperature;
  int64_t top_k;        // 0: off
  float top_p;          // 1: off
  float* logp;          // [N, V]
  uint64_t* seg_cand = nullptr;   // workspace [N, kFilterSegs, kFilterSegCap] or null
  int32_t* seg_count = nullptr;   // workspace [N, kFilterSegs]
};

// Early-determinism estimate from sampled target blocks.
struct DeterminismArgs {
  int64_t M, b, V;
  const int32_t* x;     // [M, b]
  const float* logp;    // [M, b, V]
  float* terms;         // [M]
  float* mean;          // scalar or null
};

inline int n_chunks(int nT) { return (nT + kTilesPerChunk - 1) / kTilesPerChunk; }

hipError_t launch_head(const HeadArgs& a, hipStream_t stream);
hipError_t launch_sample(const SampleArgs& a, hipStream_t stream);
hipError_t launch_verify(const VerifyArgs& a, hipStream_t stream);
hipError_t launch_sample_greedy(const GreedyArgs& a, hipStream_t stream);
hipError_t launch_verify_greedy(const GreedyArgs& a, hipStream_t stream);
hipError_t launch_objective(const ObjectiveArgs& a, hipStream_t stream);
hipError_t launch_expand(const ExpandArgs& a, hipStream_t stream);
hipError_t launch_prior_head(const PriorHeadArgs& a, hipStream_t stream);
hipError_t launch_filter(const FilterArgs& a, hipStream_t stream);
hipError_t launch_determinism(const DeterminismArgs& a, hipStream_t stream);
hipError_t launch_read_probe(const void* buf, int64_t bytes, float* partials, int64_t n_partials,
                             hipStream_t stream);

}  // namespace dbl
