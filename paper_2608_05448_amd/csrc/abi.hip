// C ABI of the DBLast library (declared in include/dblast.h): argument validation,
// workspace layout and status mapping around the kernel launchers.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <cstdio>
#include <initializer_list>
#include <mutex>
#include <string>

#include "../../include/dblast.h"
#include "kernels.hpp"

namespace {

thread_local std::string g_last_error;

dbl_status fail(dbl_status s, const std::string& msg) {
  g_last_error = std::string(dbl_status_string(s)) + ": " + msg;
  return s;
}

dbl_status ok() { return DBL_OK; }

constexpr size_t kAlign = 256;
size_t align_up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }

int64_t ntiles(int64_t V) { return (V + DBL_VTILE - 1) / DBL_VTILE; }

// Shape checks shared by every call.
dbl_status check_shape(const dbl_shape& s, bool need_d) {
  if (s.B < 0) return fail(DBL_ESHAPE, "B must be >= 0");
  if (s.K < 1 || s.R < 1 || s.V < 1) return fail(DBL_ESHAPE, "K, R and V must be >= 1");
  if (s.R > dbl::kMaxR) return fail(DBL_ESHAPE, "R must be <= 64");
  if (s.V >= (int64_t(1) << 24)) return fail(DBL_ESHAPE, "V must be < 2^24");
  if (s.K > (int64_t(1) << 20)) return fail(DBL_ESHAPE, "K must be <= 2^20");
  // The bf16 head kernels address a tile's operand rows with 32-bit byte offsets (up to 512 d).
  if (need_d && (s.d < 1 || s.d > (int64_t(1) << 20)))
    return fail(DBL_ESHAPE, "d must be in [1, 2^20]");
  const double rows = static_cast<double>(s.B) * s.K * s.R;
  if (rows * static_cast<double>(s.V) >= 4.0e18) return fail(DBL_ESHAPE, "B*K*R*V too large");
  return ok();
}

// Every array is read and written with 16-byte vector accesses, so each must be 16-byte
// aligned. NULL (an optional array that is not passed) is not checked here.
dbl_status check_aligned(std::initializer_list<std::pair<const void*, const char*>> arrays) {
  for (const auto& a : arrays)
    if (reinterpret_cast<uintptr_t>(a.first) % 16 != 0)
      return fail(DBL_EINVAL, std::string(a.second) + " is not 16-byte aligned");
  return ok();
}

struct WsLayout {
  size_t total = 0;
  size_t off[4] = {0, 0, 0, 0};
};

WsLayout layout(int op, const dbl_shape& s) {
  WsLayout L;
  const size_t B = static_cast<size_t>(s.B), K = static_cast<size_t>(s.K);
  const size_t R = static_cast<size_t>(s.R);
  const size_t nT = static_cast<size_t>(ntiles(s.V));
  const size_t nchunk = static_cast<size_t>(dbl::n_chunks(static_cast<int>(nT)));
  size_t sizes[4] = {0, 0, 0, 0};
  int n = 0;
  switch (op) {
    case DBL_OP_HEAD:  // argmax keys, used only when argmax is requested
      sizes[0] = B * K * R * sizeof(uint64_t);
      n = 1;
      break;
    case DBL_OP_SAMPLE_GREEDY:
      n = 0;
      break;
    case DBL_OP_VERIFY_GREEDY:
      sizes[0] = B * K * R * sizeof(double);
      sizes[1] = B * nT * sizeof(uint64_t);
      sizes[2] = B * nT * sizeof(uint64_t);
      n = 3;
      break;
    case DBL_OP_EXPECTED_LEN_GREEDY:
      sizes[0] = B * K * R * sizeof(double);
      n = 1;
      break;
    case DBL_OP_SAMPLE:
      n = 0;
      break;
    case DBL_OP_VERIFY:
      sizes[0] = B * K * R * sizeof(double);
      sizes[1] = B * K * nchunk * sizeof(float);
      sizes[2] = B * nT * sizeof(uint64_t);
      sizes[3] = B * nT * sizeof(uint64_t);
      n = 4;
      break;
    case DBL_OP_EXPECTED_LEN:
      sizes[0] = B * K * R * sizeof(double);
      sizes[1] = B * K * nchunk * sizeof(float);
      n = 2;
      break;
    case DBL_OP_TARGET:  // rows B*K: per-segment candidate lists and their counts
      sizes[0] = B * K * dbl::kFilterSegs * dbl::kFilterSegCap * sizeof(uint64_t);
      sizes[1] = B * K * dbl::kFilterSegs * sizeof(int32_t);
      n = 2;
      break;
    default:
      L.total = SIZE_MAX;
      return L;
  }
  size_t at = 0;
  for (int i = 0; i < n; ++i) {
    L.off[i] = at;
    at += align_up(sizes[i]);
  }
  L.total = at;
  return L;
}

dbl_status check_ws(int op, const dbl_shape& s, void* ws, size_t ws_bytes, WsLayout* out) {
  *out = layout(op, s);
  if (out->total == 0) return ok();
  if (ws == nullptr) return fail(DBL_EWORKSPACE, "workspace pointer is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0)
    return fail(DBL_EWORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < out->total)
    return fail(DBL_EWORKSPACE, "workspace has " + std::to_string(ws_bytes) + " bytes, needs " +
                                    std::to_string(out->total));
  return ok();
}

dbl_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(DBL_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

dbl::BlockArgs block_args(const dbl_shape& s, const float* tls, const float* lmass,
                          const float* lse, const float* prior, float z_temp, uint64_t seed,
                          uint64_t step, int64_t seq_offset) {
  dbl::BlockArgs a;
  a.B = s.B;
  a.K = s.K;
  a.R = s.R;
  a.V = s.V;
  a.nT = static_cast<int>(ntiles(s.V));
  a.tls = tls;
  a.lmass = lmass;
  a.lse = lse;
  a.prior = prior;
  a.z_temp = z_temp;
  a.seed = seed;
  a.step = step;
  a.seq_offset = seq_offset;
  return a;
}

dbl_status check_block_inputs(const dbl_shape& s, const float* tls, const float* lmass,
                              const float* lse, const float* prior, float z_temp) {
  if (dbl_status st = check_shape(s, false)) return st;
  if (!tls || !lmass || !lse || !prior) return fail(DBL_EINVAL, "NULL input pointer");
  if (!(z_temp >= 0.0f) || isinf(z_temp))
    return fail(DBL_EINVAL, "z_temp must be finite and >= 0");
  return check_aligned({{tls, "tls"}, {lmass, "lmass"}, {lse, "lse"}, {prior, "prior_logits"}});
}

dbl_status check_greedy_inputs(const dbl_shape& s, const int32_t* xhat, const float* prior,
                               float z_temp) {
  if (dbl_status st = check_shape(s, false)) return st;
  if (!xhat || !prior) return fail(DBL_EINVAL, "NULL input pointer");
  if (!(z_temp >= 0.0f) || isinf(z_temp))
    return fail(DBL_EINVAL, "z_temp must be finite and >= 0");
  return check_aligned({{xhat, "x_hat"}, {prior, "prior_logits"}});
}

dbl::GreedyArgs greedy_args(const dbl_shape& s, const int32_t* xhat, const float* prior,
                            float z_temp, uint64_t seed, uint64_t step, int64_t seq_offset) {
  dbl::GreedyArgs a{};
  a.blk = block_args(s, nullptr, nullptr, nullptr, prior, z_temp, seed, step, seq_offset);
  a.xhat = xhat;
  return a;
}

// Argument checks of the two verification entry points.
dbl_status check_verify(const dbl_shape& s, const float* tls, const float* lmass,
                        const float* lse, const float* prior_logits, float z_temp,
                        const int32_t* x, const float* logp, int64_t Kp, int32_t* n_accept,
                        int32_t* next_token, float* accept_mass, float* al_expected,
                        float* exp_len) {
  if (dbl_status st = check_block_inputs(s, tls, lmass, lse, prior_logits, z_temp)) return st;
  if (!x || !logp) return fail(DBL_EINVAL, "NULL input pointer");
  if (!n_accept || !next_token) return fail(DBL_EINVAL, "NULL output pointer");
  if (Kp != s.K && Kp != s.K + 1) return fail(DBL_EINVAL, "Kp must be K or K + 1");
  return check_aligned({{x, "x"}, {logp, "logp"}, {n_accept, "n_accept"},
                        {next_token, "next_token"}, {accept_mass, "accept_mass"},
                        {al_expected, "al_expected"}, {exp_len, "exp_len"}});
}

// Verification launch with its scratch carved out of `base` (a caller workspace or the fixed
// scratch) by the DBL_OP_VERIFY layout.
dbl_status launch_verify_in(const dbl_shape& s, const float* tls, const float* lmass,
                            const float* lse, const float* prior_logits, float z_temp,
                            const int32_t* x, const float* logp, int64_t Kp, uint64_t seed,
                            uint64_t step, int64_t seq_offset, int32_t* n_accept,
                            int32_t* next_token, float* accept_mass, float* al_expected,
                            float* exp_len, char* base, const WsLayout& L, void* stream) {
  dbl::VerifyArgs a;
  a.blk = block_args(s, tls, lmass, lse, prior_logits, z_temp, seed, step, seq_offset);
  a.x = x;
  a.logp = logp;
  a.Kp = Kp;
  a.trajectory = false;
  a.n_accept = n_accept;
  a.next_token = next_token;
  a.beta = accept_mass;
  a.al = al_expected;
  a.exp_len = exp_len;
  a.wpost = reinterpret_cast<double*>(base + L.off[0]);
  a.beta_part = reinterpret_cast<float*>(base + L.off[1]);
  a.res_tiles = reinterpret_cast<uint64_t*>(base + L.off[2]);
  a.p_tiles = reinterpret_cast<uint64_t*>(base + L.off[3]);
  return hip_status(dbl::launch_verify(a, static_cast<hipStream_t>(stream)), "verify launch");
}

// Scratch of dbl_verify_block_static, for callers that cannot allocate: a fixed device array,
// one copy per GPU, held until the process ends. Its name is a host-side stand-in, never a
// device address: each device's address is resolved once, with that device current, by
// hipGetSymbolAddress, and only that address is handed to kernels. Every kernel writes the
// parts it reads before reading them, so nothing needs clearing between calls.
constexpr size_t kStaticScratchBytes = size_t(8) << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

dbl_status static_scratch(void* stream, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(DBL_EHIP, "device index out of range");
  if (stream) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev);
    if (e != hipSuccess) return hip_status(e, "hipStreamGetDevice");
    if (sdev != dev) return fail(DBL_EINVAL, "stream belongs to a device other than the current one");
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!p || reinterpret_cast<uintptr_t>(p) % 256 != 0)
      return fail(DBL_EHIP, "fixed scratch has no 256-byte aligned device address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ok();
}

}  // namespace

extern "C" {

int dbl_vtile(void) { return DBL_VTILE; }

int64_t dbl_ntiles(int64_t V) { return V < 1 ? 0 : ntiles(V); }

size_t dbl_workspace_bytes(int op, dbl_shape shape) {
  if (check_shape(shape, op == DBL_OP_HEAD) != DBL_OK) return SIZE_MAX;
  return layout(op, shape).total;
}

const char* dbl_status_string(int status) {
  switch (status) {
    case DBL_OK: return "DBL_OK";
    case DBL_EINVAL: return "DBL_EINVAL";
    case DBL_ESHAPE: return "DBL_ESHAPE";
    case DBL_EDTYPE: return "DBL_EDTYPE";
    case DBL_EWORKSPACE: return "DBL_EWORKSPACE";
    case DBL_EHIP: return "DBL_EHIP";
    default: return "DBL_UNKNOWN";
  }
}

const char* dbl_last_error(void) { return g_last_error.c_str(); }

dbl_status dbl_head_logprobs(dbl_shape s, int dt, const void* h, const void* w, float* tls,
                             float* lmass, float* lse, int32_t* argmax, void* ws,
                             size_t ws_bytes, void* stream) {
  if (dbl_status st = check_shape(s, true)) return st;
  if (dt != DBL_F32 && dt != DBL_BF16) return fail(DBL_EDTYPE, "dtype must be DBL_F32 or DBL_BF16");
  if (dt == DBL_BF16 && s.d % 8 != 0) return fail(DBL_ESHAPE, "bf16 head needs d % 8 == 0");
  if (!h || !w || !tls || !lmass || !lse) return fail(DBL_EINVAL, "NULL pointer");
  if (dbl_status st = check_aligned({{h, "h"}, {w, "w"}, {tls, "tls"}, {lmass, "lmass"},
                                     {lse, "lse"}, {argmax, "argmax"}}))
    return st;
  WsLayout L;
  if (argmax) {
    if (dbl_status st = check_ws(DBL_OP_HEAD, s, ws, ws_bytes, &L)) return st;
  }
  if (s.B == 0) return ok();
  dbl::HeadArgs a;
  a.M = s.B * s.K * s.R;
  a.V = s.V;
  a.d = static_cast<int>(s.d);
  a.dtype_bf16 = dt == DBL_BF16;
  a.h = h;
  a.w = w;
  a.tls = tls;
  a.lmass = lmass;
  a.lse = lse;
  a.argmax = argmax;
  a.amax_keys = argmax ? reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + L.off[0]) : nullptr;
  return hip_status(dbl::launch_head(a, static_cast<hipStream_t>(stream)), "head launch");
}

dbl_status dbl_sample_block(dbl_shape s, const float* tls, const float* lmass,
                            const float* lse, const float* prior_logits, float z_temp,
                            uint64_t seed, uint64_t step, int64_t seq_offset, int32_t* z_out,
                            int32_t* x_out, void* ws, size_t ws_bytes, void* stream) {
  if (dbl_status st = check_block_inputs(s, tls, lmass, lse, prior_logits, z_temp)) return st;
  if (!z_out || !x_out) return fail(DBL_EINVAL, "NULL output pointer");
  if (dbl_status st = check_aligned({{z_out, "z_out"}, {x_out, "x_out"}})) return st;
  WsLayout L;
  if (dbl_status st = check_ws(DBL_OP_SAMPLE, s, ws, ws_bytes, &L)) return st;
  if (s.B == 0) return ok();
  dbl::SampleArgs a;
  a.blk = block_args(s, tls, lmass, lse, prior_logits, z_temp, seed, step, seq_offset);
  a.z_out = z_out;
  a.x_out = x_out;
  return hip_status(dbl::launch_sample(a, static_cast<hipStream_t>(stream)), "sample launch");
}

dbl_status dbl_verify_block(dbl_shape s, const float* tls, const float* lmass,
                            const float* lse, const float* prior_logits, float z_temp,
                            const int32_t* x, const float* logp, int64_t Kp, uint64_t seed,
                            uint64_t step, int64_t seq_offset, int32_t* n_accept,
                            int32_t* next_token, float* accept_mass, float* al_expected,
                            float* exp_len, void* ws, size_t ws_bytes, void* stream) {
  if (dbl_status st = check_verify(s, tls, lmass, lse, prior_logits, z_temp, x, logp, Kp,
                                   n_accept, next_token, accept_mass, al_expected, exp_len))
    return st;
  WsLayout L;
  if (dbl_status st = check_ws(DBL_OP_VERIFY, s, ws, ws_bytes, &L)) return st;
  if (s.B == 0) return ok();
  return launch_verify_in(s, tls, lmass, lse, prior_logits, z_temp, x, logp, Kp, seed, step,
                          seq_offset, n_accept, next_token, accept_mass, al_expected, exp_len,
                          static_cast<char*>(ws), L, stream);
}

dbl_status dbl_verify_block_static(dbl_shape s, const float* tls, const float* lmass,
                                   const float* lse, const float* prior_logits, float z_temp,
                                   const int32_t* x, const float* logp, int64_t Kp,
                                   uint64_t seed, uint64_t step, int64_t seq_offset,
                                   int32_t* n_accept, int32_t* next_token, float* accept_mass,
                                   float* al_expected, float* exp_len, void* stream) {
  if (dbl_status st = check_verify(s, tls, lmass, lse, prior_logits, z_temp, x, logp, Kp,
                                   n_accept, next_token, accept_mass, al_expected, exp_len))
    return st;
  const WsLayout L = layout(DBL_OP_VERIFY, s);
  if (L.total > kStaticScratchBytes)
    return fail(DBL_EWORKSPACE, "this shape needs " + std::to_string(L.total) +
                                    " bytes of scratch; the fixed scratch holds " +
                                    std::to_string(kStaticScratchBytes));
  if (s.B == 0) return ok();
  void* base = nullptr;
  if (dbl_status st = static_scratch(stream, &base)) return st;
  return launch_verify_in(s, tls, lmass, lse, prior_logits, z_temp, x, logp, Kp, seed, step,
                          seq_offset, n_accept, next_token, accept_mass, al_expected, exp_len,
                          static_cast<char*>(base), L, stream);
}

dbl_status dbl_expected_len(dbl_shape s, const float* tls, const float* lmass,
                            const float* lse, const float* prior_logits, float z_temp,
                            const int32_t* x, const float* logp, float* beta, float* exp_len,
                            void* ws, size_t ws_bytes, void* stream) {
  if (dbl_status st = check_block_inputs(s, tls, lmass, lse, prior_logits, z_temp)) return st;
  if (!x || !logp) return fail(DBL_EINVAL, "NULL input pointer");
  if (!exp_len) return fail(DBL_EINVAL, "NULL output pointer");
  if (dbl_status st = check_aligned({{x, "x"}, {logp, "logp"}, {beta, "beta"},
                                     {exp_len, "exp_len"}}))
    return st;
  WsLayout L;
  if (dbl_status st = check_ws(DBL_OP_EXPECTED_LEN, s, ws, ws_bytes, &L)) return st;
  if (s.B == 0) return ok();
  char* base = static_cast<char*>(ws);
  dbl::VerifyArgs a;
  a.blk = block_args(s, tls, lmass, lse, prior_logits, z_temp, 0, 0, 0);
  a.x = x;
  a.logp = logp;
  a.Kp = s.K;
  a.trajectory = true;
  a.n_accept = nullptr;
  a.next_token = nullptr;
  a.beta = beta;
  a.al = nullptr;
  a.exp_len = exp_len;
  a.wpost = reinterpret_cast<double*>(base + L.off[0]);
  a.beta_part = reinterpret_cast<float*>(base + L.off[1]);
  a.res_tiles = nullptr;
  a.p_tiles = nullptr;
  return hip_status(dbl::launch_verify(a, static_cast<hipStream_t>(stream)),
                    "expected_len launch");
}

dbl_status dbl_sample_greedy(dbl_shape s, const int32_t* x_hat, const float* prior_logits,
                             float z_temp, uint64_t seed, uint64_t step, int64_t seq_offset,
                             int32_t* z_out, int32_t* x_out, void* stream) {
  if (dbl_status st = check_greedy_inputs(s, x_hat, prior_logits, z_temp)) return st;
  if (!z_out || !x_out) return fail(DBL_EINVAL, "NULL output pointer");
  if (dbl_status st = check_aligned({{z_out, "z_out"}, {x_out, "x_out"}})) return st;
  if (s.B == 0) return ok();
  dbl::GreedyArgs a = greedy_args(s, x_hat, prior_logits, z_temp, seed, step, seq_offset);
  a.z_out = z_out;
  a.x_out = x_out;
  return hip_status(dbl::launch_sample_greedy(a, static_cast<hipStream_t>(stream)),
                    "greedy sample launch");
}

dbl_status dbl_verify_greedy(dbl_shape s, const int32_t* x_hat, const float* prior_logits,
                             float z_temp, const int32_t* x, const float* logp, int64_t Kp,
                             uint64_t seed, uint64_t step, int64_t seq_offset, int32_t* n_accept,
                             int32_t* next_token, float* accept_mass, float* al_expected,
                             float* exp_len, void* ws, size_t ws_bytes, void* stream) {
  if (dbl_status st = check_greedy_inputs(s, x_hat, prior_logits, z_temp)) return st;
  if (!x || !logp) return fail(DBL_EINVAL, "NULL input pointer");
  if (!n_accept || !next_token) return fail(DBL_EINVAL, "NULL output pointer");
  if (Kp != s.K && Kp != s.K + 1) return fail(DBL_EINVAL, "Kp must be K or K + 1");
  if (dbl_status st = check_aligned({{x, "x"}, {logp, "logp"}, {n_accept, "n_accept"},
                                     {next_token, "next_token"}, {accept_mass, "accept_mass"},
                                     {al_expected, "al_expected"}, {exp_len, "exp_len"}}))
    return st;
  WsLayout L;
  if (dbl_status st = check_ws(DBL_OP_VERIFY_GREEDY, s, ws, ws_bytes, &L)) return st;
  if (s.B == 0) return ok();
  char* base = static_cast<char*>(ws);
  dbl::GreedyArgs a = greedy_args(s, x_hat, prior_logits, z_temp, seed, step, seq_offset);
  a.x = x;
  a.logp = logp;
  a.Kp = Kp;
  a.trajectory = false;
  a.n_accept = n_accept;
  a.next_token = next_token;
  a.beta = accept_mass;
  a.al = al_expected;
  a.exp_len = exp_len;
  a.wpost = reinterpret_cast<double*>(base + L.off[0]);
  a.res_tiles = reinterpret_cast<uint64_t*>(base + L.off[1]);
  a.p_tiles = reinterpret_cast<uint64_t*>(base + L.off[2]);
  return hip_status(dbl::launch_verify_greedy(a, static_cast<hipStream_t>(stream)),
                    "greedy verify launch");
}

dbl_status dbl_expected_len_greedy(dbl_shape s, const int32_t* x_hat,
                                   const float* prior_logits, float z_temp, const int32_t* x,
                                   const float* logp, float* beta, float* exp_len, void* ws,
                                   size_t ws_bytes, void* stream) {
  if (dbl_status st = check_greedy_inputs(s, x_hat, prior_logits, z_temp)) return st;
  if (!x || !logp) return fail(DBL_EINVAL, "NULL input pointer");
  if (!exp_len) return fail(DBL_EINVAL, "NULL output pointer");
  if (dbl_status st = check_aligned({{x, "x"}, {logp, "logp"}, {beta, "beta"},
                                     {exp_len, "exp_len"}}))
    return st;
  WsLayout L;
  if (dbl_status st = check_ws(DBL_OP_EXPECTED_LEN_GREEDY, s, ws, ws_bytes, &L)) return st;
  if (s.B == 0) return ok();
  dbl::GreedyArgs a = greedy_args(s, x_hat, prior_logits, z_temp, 0, 0, 0);
  a.x = x;
  a.logp = logp;
  a.Kp = s.K;
  a.trajectory = true;
  a.beta = beta;
  a.exp_len = exp_len;
  a.wpost = reinterpret_cast<double*>(static_cast<char*>(ws) + L.off[0]);
  return hip_status(dbl::launch_verify_greedy(a, static_cast<hipStream_t>(stream)),
                    "greedy expected_len launch");
}

dbl_status dbl_acceptance_objective(dbl_shape s, const float* tls, const float* lmass,
                                    const float* lse, const float* prior_logits, float z_temp,
                                    const int32_t* x, const float* logp, float tau, float* log_r,
                                    float* S, int32_t* ell_tau, float* J, float* nll,
                                    void* stream) {
  if (dbl_status st = check_block_inputs(s, tls, lmass, lse, prior_logits, z_temp)) return st;
  if (!x || !logp) return fail(DBL_EINVAL, "NULL input pointer");
  if (!ell_tau || !J || !nll) return fail(DBL_EINVAL, "NULL output pointer");
  if (!(tau > 0.0f) || isinf(tau)) return fail(DBL_EINVAL, "tau must be finite and > 0");
  if (dbl_status st = check_aligned({{x, "x"}, {logp, "logp"}, {log_r, "log_r"}, {S, "S"},
                                     {ell_tau, "ell_tau"}, {J, "J"}, {nll, "nll"}}))
    return st;
  if (s.B == 0) return ok();
  dbl::ObjectiveArgs a{};
  a.blk = block_args(s, tls, lmass, lse, prior_logits, z_temp, 0, 0, 0);
  a.x = x;
  a.logp = logp;
  a.tau = tau;
  a.log_r = log_r;
  a.S = S;
  a.ell_tau = ell_tau;
  a.J = J;
  a.nll = nll;
  return hip_status(dbl::launch_objective(a, static_cast<hipStream_t>(stream)),
                    "objective launch");
}

dbl_status dbl_expand_branches(dbl_shape s, const void* h, const void* W, const void* c,
                               void* h_out, void* stream) {
  if (s.B < 0 || s.K < 1 || s.R < 1 || s.R > dbl::kMaxR)
    return fail(DBL_ESHAPE, "need B >= 0, K >= 1 and 1 <= R <= 64");
  if (s.d < 32 || s.d % 32 != 0 || s.d > (int64_t(1) << 20))
    return fail(DBL_ESHAPE, "expander needs d % 32 == 0 and 32 <= d <= 2^20");
  if (static_cast<double>(s.B) * s.K * s.R * s.d >= 4.0e18)
    return fail(DBL_ESHAPE, "B*K*R*d too large");
  if (!h || !W || !c || !h_out) return fail(DBL_EINVAL, "NULL pointer");
  if (dbl_status st = check_aligned({{h, "h"}, {W, "W"}, {c, "c"}, {h_out, "h_out"}}))
    return st;
  if (s.B == 0) return ok();
  dbl::ExpandArgs a;
  a.M = s.B * s.K;
  a.R = s.R;
  a.d = static_cast<int>(s.d);
  a.h = h;
  a.W = W;
  a.c = c;
  a.out = h_out;
  return hip_status(dbl::launch_expand(a, static_cast<hipStream_t>(stream)), "expander launch");
}

dbl_status dbl_prior_head(dbl_shape s, const void* h_anchor, const void* U, const void* e,
                          float* prior_logits, void* stream) {
  if (s.B < 0 || s.R < 1 || s.R > dbl::kMaxR || s.d < 1 || s.d > (int64_t(1) << 30))
    return fail(DBL_ESHAPE, "need B >= 0, 1 <= R <= 64 and 1 <= d <= 2^30");
  if (!h_anchor || !U || !e || !prior_logits) return fail(DBL_EINVAL, "NULL pointer");
  if (dbl_status st = check_aligned({{h_anchor, "h_anchor"}, {U, "U"}, {e, "e"},
                                     {prior_logits, "prior_logits"}}))
    return st;
  if (s.B == 0) return ok();
  dbl::PriorHeadArgs a;
  a.B = s.B;
  a.R = static_cast<int>(s.R);
  a.d = static_cast<int>(s.d);
  a.h_anchor = h_anchor;
  a.U = U;
  a.e = e;
  a.ell = prior_logits;
  return hip_status(dbl::launch_prior_head(a, static_cast<hipStream_t>(stream)),
                    "prior head launch");
}

dbl_status dbl_target_logprobs(int64_t N, int64_t V, const float* logits, float temperature,
                               int64_t top_k, float top_p, float* logp, void* ws,
                               size_t ws_bytes, void* stream) {
  if (N < 0 || V < 1 || V >= (int64_t(1) << 24)) return fail(DBL_ESHAPE, "need N >= 0, 1 <= V < 2^24");
  if (static_cast<double>(N) * static_cast<double>(V) >= 4.0e18)
    return fail(DBL_ESHAPE, "N*V too large");
  if (!logits || !logp) return fail(DBL_EINVAL, "NULL pointer");
  if (dbl_status st = check_aligned({{logits, "logits"}, {logp, "logp"}})) return st;
  {
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(logits), b0 = reinterpret_cast<uintptr_t>(logp);
    const uintptr_t len = static_cast<uintptr_t>(N) * static_cast<uintptr_t>(V) * sizeof(float);
    if (len > 0 && a0 < b0 + len && b0 < a0 + len)
      return fail(DBL_EINVAL, "logp must not overlap logits");
  }
  if (!(temperature >= 0.0f) || isinf(temperature))
    return fail(DBL_EINVAL, "temperature must be finite and >= 0");
  if (top_k < 0) return fail(DBL_EINVAL, "top_k must be >= 0");
  if (!(top_p > 0.0f && top_p <= 1.0f)) return fail(DBL_EINVAL, "top_p must be in (0, 1]");
  WsLayout L;
  const bool use_ws = ws != nullptr || ws_bytes != 0;
  if (use_ws) {
    const dbl_shape rows{N, 1, 1, 0, V};
    if (dbl_status st = check_ws(DBL_OP_TARGET, rows, ws, ws_bytes, &L)) return st;
  }
  if (N == 0) return ok();
  dbl::FilterArgs a;
  a.N = N;
  a.V = V;
  a.logits = logits;
  a.temperature = temperature;
  a.top_k = top_k;
  a.top_p = top_p;
  a.logp = logp;
  if (use_ws) {
    a.seg_cand = reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + L.off[0]);
    a.seg_count = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + L.off[1]);
  }
  return hip_status(dbl::launch_filter(a, static_cast<hipStream_t>(stream)), "filter launch");
}

dbl_status dbl_early_determinism(int64_t M, int64_t b, int64_t V, const int32_t* x,
                                 const float* logp, float* terms, float* mean, void* stream) {
  if (M < 0 || b < 1 || V < 1 || V >= (int64_t(1) << 24))
    return fail(DBL_ESHAPE, "need M >= 0, b >= 1, 1 <= V < 2^24");
  if (static_cast<double>(M) * b * V >= 4.0e18) return fail(DBL_ESHAPE, "M*b*V too large");
  if (!x || !logp || !terms) return fail(DBL_EINVAL, "NULL pointer");
  if (dbl_status st = check_aligned({{x, "x"}, {logp, "logp"}, {terms, "terms"}, {mean, "mean"}}))
    return st;
  if (M == 0) return ok();
  dbl::DeterminismArgs a;
  a.M = M;
  a.b = b;
  a.V = V;
  a.x = x;
  a.logp = logp;
  a.terms = terms;
  a.mean = mean;
  return hip_status(dbl::launch_determinism(a, static_cast<hipStream_t>(stream)),
                    "early determinism launch");
}

dbl_status dbl_stream_read_probe(const void* buf, int64_t bytes, float* partials,
                                 int64_t n_partials, void* stream) {
  if (!buf || !partials) return fail(DBL_EINVAL, "NULL pointer");
  if (bytes < 0 || bytes % 16 != 0) return fail(DBL_ESHAPE, "bytes must be a multiple of 16");
  if (n_partials < 1 || n_partials > (int64_t(1) << 20))
    return fail(DBL_ESHAPE, "need 1 <= n_partials <= 2^20");
  if (dbl_status st = check_aligned({{buf, "buf"}, {partials, "partials"}})) return st;
  return hip_status(dbl::launch_read_probe(buf, bytes, partials, n_partials,
                                           static_cast<hipStream_t>(stream)),
                    "read probe launch");
}

}  // extern "C"
