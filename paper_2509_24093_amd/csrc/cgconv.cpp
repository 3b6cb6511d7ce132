// Plan and C ABI of the global CG convolution (see include/cgconv.h).
//
// Forward pipeline for one call, all on the caller's stream:
//   N <= 256 : DFT(z = q + i k) -> CG stage -> inverse DFT (x 1/N, split)
//   N  > 256 : N = N1 * N2 four-step factorisation with n = n2 + N2 n1 and
//              w = w1 + N1 w2:
//     F1  for each n2: length-N1 DFT over n1, twiddle W_N^(n2 w1)   q,k -> Y
//     F2  for each w1: length-N2 DFT over n2                         Y -> Z
//         (Z, W keep frequency w1 + N1 w2 at row w1 N2 + w2, so F2 and I1
//          read and write contiguous row blocks)
//     CG  sparse tensor product per frequency pair and channel       Z -> W
//     I1  for each w1: inverse length-N2 DFT, twiddle W_N^(-n2 w1)   W -> V
//     I2  for each n2: inverse length-N1 DFT, x 1/N, split channels  V -> out
// Y, Z, W, V live in two plan-owned workspaces of B*N*K*C float2 each.
//   512 <= N <= 32768, L_max <= 6: N2 = 64 and F2 + CG + I1 run as one fused
//   kernel (cg_fused.hip) between F1 and I2; the spectra stay on chip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <complex>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "cgconv.h"
#include "cg_table.h"
#include "gate_bwd.h"
#include "gft.h"
#include "kernels.h"

using namespace cgconv;

namespace {

thread_local std::string g_last_error;

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
}

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }
int ilog2(int64_t x) {
  int r = 0;
  while ((int64_t(1) << r) < x) ++r;
  return r;
}

}  // namespace

struct cgconv_plan {
  int64_t B = 0, N = 0, C = 0, Cp = 0;  // N: length of the token DFTs
  int64_t Nu = 0;                        // tokens of the caller's arrays (= N, or fewer with zero padding)
  bool linear = false;                   // zero-padded token boundary
  bool graph = false;                    // graph Fourier plan (cgconv_forward_graph only)
  // graph plans: padded sizes and the split operands of the two transforms
  int64_t Kp = 0, Mp = 0, KCp = 0;
  uint16_t *ga_fh = nullptr, *ga_fl = nullptr, *ga_ih = nullptr, *ga_il = nullptr;  // U^T and U, [B][Mp][Kp]
  uint16_t *gb_fh = nullptr, *gb_fl = nullptr;  // [q | k]^T, [B][2 KCp][Kp]
  uint16_t *gb_ih = nullptr, *gb_il = nullptr;  // u_hat^T, [B][KCp][Kp]
  float* g_spec = nullptr;                      // [q_hat | k_hat], [B][n][2 KCp]
  float* g_uhat = nullptr;                      // [B][n][K C]
  void* g_block = nullptr;                      // one allocation holding all of the above
  int L = 0, K = 0;
  int64_t N1 = 0, N2 = 0;  // N1 == 0: single pass
  bool fused = false;      // two-pass with N2 = 64 and the fused middle kernel
  bool small = false;      // DFT length <= 256: the forward is one block per channel group (cg_small.hip)
  int small_cc = 0, small_threads = 0;
  int device = 0;
  int64_t nnz = 0, paths = 0, products = 0;  // nnz: complex-basis terms the contraction evaluates
  // the real-basis tensor the plan's kernels evaluate (cgconv_plan_export_table)
  std::vector<RealEntry> rtable;
  size_t ws_bytes = 0;
  float2* tw = nullptr;
  float2* ws1 = nullptr;
  float2* ws2 = nullptr;
  int* d_offs = nullptr;
  uint32_t* d_tkey = nullptr;
  float* d_tcoef = nullptr;
  uint16_t* d_wmix = nullptr;  // channel-mixing weights, split bf16 MFMA operands (L <= 6, C <= 32)
  float2* d_gpart = nullptr;   // gating: online-softmax partials per token chunk
  float2* d_gfin = nullptr;    // gating: maximum and denominator per (b, l, c)
  float* d_gh = nullptr;       // gating backward: h per (b, i, l, c)
  float* d_gS = nullptr;       // gating backward: sum of h over the tokens per (b, l, c)
  float* d_bscale = nullptr;   // backward: per-component scales, [2 gradients][in a, in b, out][K]
  bool force_generic = false;
  // optional per-stage timing: events recorded on the forward's stream.  The
  // first timed call fixes the kind (plain or mixed) that is timed.
  int n_stages = 0, n_stages_mix = 0;
  int timing_max = 0, timing_calls = 0, timing_kind = -1;
  std::vector<hipEvent_t> events;  // timing_max * kMaxEvents
};

namespace {

void free_plan(cgconv_plan* p) {
  if (!p) return;
  int cur = 0;
  (void)hipGetDevice(&cur);
  (void)hipSetDevice(p->device);
  (void)hipFree(p->tw);
  (void)hipFree(p->ws1);
  (void)hipFree(p->ws2);
  (void)hipFree(p->d_offs);
  (void)hipFree(p->d_tkey);
  (void)hipFree(p->d_tcoef);
  (void)hipFree(p->d_wmix);
  (void)hipFree(p->d_gpart);
  (void)hipFree(p->d_gfin);
  (void)hipFree(p->d_gh);
  (void)hipFree(p->d_gS);
  (void)hipFree(p->d_bscale);
  (void)hipFree(p->g_block);
  for (hipEvent_t ev : p->events) (void)hipEventDestroy(ev);
  (void)hipSetDevice(cur);
  delete p;
}

const char* const kStages2[] = {"fft_fwd_1", "fft_fwd_2", "cg", "fft_inv_1", "fft_inv_2"};
const char* const kStages1[] = {"fft_fwd", "cg", "fft_inv"};
const char* const kStagesF[] = {"fft_fwd_1", "cg_fused", "fft_inv_2"};
const char* const kStagesS[] = {"cg_small"};
const char* const kStagesM2[] = {"fft_fwd_1", "fft_fwd_2", "cg_mix", "fft_inv_1", "fft_inv_2"};
const char* const kStagesM1[] = {"fft_fwd", "cg_mix", "fft_inv"};
const char* const kStagesG[] = {"gate_partials", "gate_finalize", "gate_value"};
const char* const kStagesGB[] = {"gate_stats", "gate_bwd", "gate_sums", "gate_bwd_du"};
const char* const kStagesI2[] = {"fft_fwd_1", "fft_fwd_2", "cg_inter", "fft_inv_1", "fft_inv_2"};
const char* const kStagesI1[] = {"fft_fwd", "cg_inter", "fft_inv"};
const char* const kStagesGft[] = {"gft_split_u", "gft_split_x", "gft_gemm_fwd", "gft_product", "gft_split_uhat",
                                  "gft_gemm_inv"};
// timing kinds: 0 forward, 1 mixed forward, 2 backward (each gradient one call), 3 gating, 4 graph forward,
// 5 gating backward
constexpr int kKindGate = 3;
constexpr int kKindGateBwd = 5;
constexpr int kKindGraph = 4;
constexpr int kKindInter = 6;
constexpr int kKindSmall = 7;
constexpr int kMaxEvents = 8;  // stages + 1 of the longest pipeline

hipError_t launch_product(int L, const GftProductArgs& a, hipStream_t s) {
  switch (L) {
    case 0: return launch_gft_product<0>(a, s);
    case 1: return launch_gft_product<1>(a, s);
    case 2: return launch_gft_product<2>(a, s);
    case 3: return launch_gft_product<3>(a, s);
    case 4: return launch_gft_product<4>(a, s);
    case 5: return launch_gft_product<5>(a, s);
    case 6: return launch_gft_product<6>(a, s);
    case 7: return launch_gft_product<7>(a, s);
    case 8: return launch_gft_product<8>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gate(int L, const GateArgs& a, hipStream_t s) {
  switch (L) {
    case 0: return launch_gate_value<0>(a, s);
    case 1: return launch_gate_value<1>(a, s);
    case 2: return launch_gate_value<2>(a, s);
    case 3: return launch_gate_value<3>(a, s);
    case 4: return launch_gate_value<4>(a, s);
    case 5: return launch_gate_value<5>(a, s);
    case 6: return launch_gate_value<6>(a, s);
    case 7: return launch_gate_value<7>(a, s);
    case 8: return launch_gate_value<8>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gate_bwd(int L, const GateBwdArgs& a, hipStream_t s) {
  switch (L) {
    case 0: return launch_gate_backward<0>(a, s);
    case 1: return launch_gate_backward<1>(a, s);
    case 2: return launch_gate_backward<2>(a, s);
    case 3: return launch_gate_backward<3>(a, s);
    case 4: return launch_gate_backward<4>(a, s);
    case 5: return launch_gate_backward<5>(a, s);
    case 6: return launch_gate_backward<6>(a, s);
    case 7: return launch_gate_backward<7>(a, s);
    case 8: return launch_gate_backward<8>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_mix(int L, const CgArgs& a, hipStream_t s) {
  switch (L) {
    case 0: return launch_cg_mix<0>(a, s);
    case 1: return launch_cg_mix<1>(a, s);
    case 2: return launch_cg_mix<2>(a, s);
    case 3: return launch_cg_mix<3>(a, s);
    case 4: return launch_cg_mix<4>(a, s);
    case 5: return launch_cg_mix<5>(a, s);
    case 6: return launch_cg_mix<6>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_inter(int L, const InterArgs& a, hipStream_t s) {
  switch (L) {
    case 0: return launch_cg_inter<0>(a, s);
    case 1: return launch_cg_inter<1>(a, s);
    case 2: return launch_cg_inter<2>(a, s);
    case 3: return launch_cg_inter<3>(a, s);
    case 4: return launch_cg_inter<4>(a, s);
    case 5: return launch_cg_inter<5>(a, s);
    case 6: return launch_cg_inter<6>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_small(int L, const SmallArgs& a, hipStream_t s) {
  switch (L) {
    case 0: return launch_cg_small<0>(a, s);
    case 1: return launch_cg_small<1>(a, s);
    case 2: return launch_cg_small<2>(a, s);
    case 3: return launch_cg_small<3>(a, s);
    case 4: return launch_cg_small<4>(a, s);
    case 5: return launch_cg_small<5>(a, s);
    case 6: return launch_cg_small<6>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t prepare_small(int L, int lds_bytes) {
  switch (L) {
    case 0: return prepare_cg_small<0>(lds_bytes);
    case 1: return prepare_cg_small<1>(lds_bytes);
    case 2: return prepare_cg_small<2>(lds_bytes);
    case 3: return prepare_cg_small<3>(lds_bytes);
    case 4: return prepare_cg_small<4>(lds_bytes);
    case 5: return prepare_cg_small<5>(lds_bytes);
    case 6: return prepare_cg_small<6>(lds_bytes);
    default: return hipErrorInvalidValue;
  }
}

// LDS bytes of the one-block kernel for cc channels per block
int64_t small_lds_bytes(int64_t Nf, int K, int cc) { return (Nf * K * cc + Nf) * 8; }

hipError_t launch_fused(int L, const FusedArgs& a, hipStream_t s) {
  switch (L) {
    case 0: return launch_cg_fused<0>(a, s);
    case 1: return launch_cg_fused<1>(a, s);
    case 2: return launch_cg_fused<2>(a, s);
    case 3: return launch_cg_fused<3>(a, s);
    case 4: return launch_cg_fused<4>(a, s);
    case 5: return launch_cg_fused<5>(a, s);
    case 6: return launch_cg_fused<6>(a, s);
    default: return hipErrorInvalidValue;
  }
}

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

template <class T>
hipError_t upload(T** dst, const std::vector<T>& src) {
  hipError_t e = hipMalloc(reinterpret_cast<void**>(dst), src.size() * sizeof(T));
  if (e != hipSuccess) return e;
  return hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice);
}

PassArgs base_args(const cgconv_plan* p) {
  PassArgs a;
  std::memset(&a, 0, sizeof a);
  a.tw = p->tw;
  a.C = (int)p->C;
  a.Cp = (int)p->Cp;
  a.KC = (int)(p->K * p->C);
  a.Nmask = (int)(p->N - 1);
  a.scale = 1.0f;
  a.in_rows = (int)p->Nu;
  a.out_rows = (int)p->Nu;
  return a;
}

// weights != nullptr: the channel-mixing stage with the unfused passes.
// scales != nullptr (fp32 only): the adjoint form used by the backward,
//   out = s_o * conv(s_a * q, s_b * reverse(k)), reverse(k)[n] = k[-n mod N],
// with per-component scales s_a = scales[0..K), s_b = scales[K..2K),
// s_o = scales[2K..3K) (device memory), applied in the first and last passes.
int run_forward(cgconv_plan* p, const void* q, const void* k, void* out, bool bf16, hipStream_t s,
                const float* weights = nullptr, const float* scales = nullptr) {
  const bool mix = weights != nullptr;
  const int K = p->K;
  const long long Wz = (long long)K * p->C;   // complex columns of z
  const long long Ww = (long long)K * p->Cp;  // complex columns of the packed output spectra
  const int in_pair = (scales ? IN_PAIR_F32_SCALED_REV : (bf16 ? IN_PAIR_BF16 : IN_PAIR_F32)) + (p->linear ? 3 : 0);
  const int out_split = scales ? OUT_SPLIT_F32_SCALED : (bf16 ? OUT_SPLIT_BF16 : OUT_SPLIT_F32);
  hipError_t e;
  auto pass = [&](int R, int inm, int outm, int dir, int groups, const void* in0, const void* in1, void* o,
                  long long ib, long long ob, int W, int gs_in, int es_in, int gs_out, int fs_out, int inter,
                  float scale) {
    PassDesc d;
    d.R = R;
    d.in_mode = inm;
    d.out_mode = outm;
    d.dir = dir;
    d.groups = groups;
    d.batch = (int)p->B;
    d.a = base_args(p);
    d.a.in0 = in0;
    d.a.in1 = in1;
    d.a.out = o;
    d.a.in_bstride = ib;
    d.a.out_bstride = ob;
    d.a.W = W;
    d.a.gs_in = gs_in;
    d.a.es_in = es_in;
    d.a.gs_out = gs_out;
    d.a.fs_out = fs_out;
    d.a.tw_stride = (int)(p->N / R);
    d.a.inter = inter;
    d.a.scale = scale;
    if (scales) {
      d.a.in_scale = scales;
      d.a.out_scale = scales + 2 * K;
    }
    return launch_fft_pass(d, s);
  };
  CgArgs ca;
  ca.N = p->N;
  ca.F = p->N / 2 + 1;
  ca.K = K;
  ca.C = (int)p->C;
  ca.Cp = (int)p->Cp;
  ca.npts = p->B * ca.F * 2 * p->Cp;
  ca.offs = p->d_offs;
  ca.tkey = p->d_tkey;
  ca.tcoef = p->d_tcoef;
  ca.wmix = p->d_wmix;
  ca.n1_log2 = ilog2(p->N1 ? p->N1 : p->N);
  ca.n2_log2 = ilog2(p->N1 ? p->N2 : 1);
  const long long N = p->N;
  const long long Nu = p->Nu;  // rows of q, k and out (padded rows are implicit zeros)
  const float inv_n = 1.0f / (float)N;
  hipEvent_t* ev = nullptr;  // events of this call if it is timed
  const bool small = p->small && !mix && !scales;
  const int kind = mix ? 1 : (scales ? 2 : (small ? kKindSmall : 0));  // 2: one half of a backward
  if (p->timing_calls < p->timing_max && (p->timing_kind < 0 || p->timing_kind == kind)) {
    p->timing_kind = kind;
    ev = &p->events[(size_t)p->timing_calls * kMaxEvents];
    ++p->timing_calls;
  }
  int stage = 0;
  auto mark = [&]() {
    if (ev) (void)hipEventRecord(ev[stage], s);
    ++stage;
  };
  mark();
  if (mix) {
    e = launch_prepare_mix_weights(weights, p->d_wmix, (int)p->paths, (int)p->C, s);
    if (e != hipSuccess) goto fail;
  }
  if (small) {
    // the whole convolution in one kernel: load, DFT, contraction, inverse
    // DFT and store per (batch element, channel group), spectra in LDS
    SmallArgs sa;
    sa.q = q;
    sa.k = k;
    sa.out = out;
    sa.tw = p->tw;
    sa.B = (int)p->B;
    sa.C = (int)p->C;
    sa.Nf = (int)N;
    sa.lg = ilog2(N);
    sa.in_rows = (int)Nu;
    sa.out_rows = (int)Nu;
    sa.cc = p->small_cc;
    sa.lcc = ilog2(p->small_cc);
    sa.mz = 0xFFFFFFFFu / (uint32_t)(K * p->small_cc) + 1;
    sa.mv = 0xFFFFFFFFu / (uint32_t)(K * p->small_cc / 2) + 1;
    sa.groups = (int)((p->C + p->small_cc - 1) / p->small_cc);
    sa.threads = p->small_threads;
    sa.bf16 = bf16;
    e = launch_small(p->L, sa, s);
    if (e != hipSuccess) goto fail;
    mark();
  } else if (p->fused && !mix) {
    // F1 (Y rows w1*64 + n2) -> fused F2 + CG + I1 (V rows w1*64 + n2) -> I2
    const int N1 = (int)p->N1, N2 = 64;
    e = pass(N1, in_pair, OUT_COMPLEX, -1, N2, q, k, p->ws1, Nu * Wz, N * Wz, (int)Wz, 1, N2, 1, N2, 1, 1.0f);
    if (e != hipSuccess) goto fail;
    mark();
    FusedArgs fa;
    fa.Y = p->ws1;
    fa.V = p->ws2;
    fa.tw = p->tw;
    fa.N = N;
    fa.N1 = N1;
    fa.units = N1 / 2 + 1;
    fa.B = (int)p->B;
    fa.C = (int)p->C;
    fa.Cp = (int)p->Cp;
    fa.Cb = (int)((p->C + 3) / 4);
    e = launch_fused(p->L, fa, s);
    if (e != hipSuccess) goto fail;
    mark();
    e = pass(N1, IN_COMPLEX, out_split, 1, N2, p->ws2, nullptr, out, N * Ww, Nu * K * p->C, (int)Ww, 1, N2, 1, N2, 0,
             inv_n);
    if (e != hipSuccess) goto fail;
    mark();
  } else if (p->N1 == 0) {
    e = pass((int)N, in_pair, OUT_COMPLEX, -1, 1, q, k, p->ws1, Nu * Wz, N * Wz, (int)Wz, 0, 1, 0, 1, 0, 1.0f);
    if (e != hipSuccess) goto fail;
    mark();
    ca.Z = p->ws1;
    ca.W = p->ws2;
    ca.trash = p->ws2 + p->B * N * K * p->Cp;
    e = mix ? launch_mix(p->L, ca, s) : launch_cg(p->L, ca, p->force_generic, s);
    if (e != hipSuccess) goto fail;
    mark();
    e = pass((int)N, IN_COMPLEX, out_split, 1, 1, p->ws2, nullptr, out, N * Ww, Nu * K * p->C, (int)Ww, 0, 1, 0, 1,
             0, inv_n);
    if (e != hipSuccess) goto fail;
    mark();
  } else {
    const int N1 = (int)p->N1, N2 = (int)p->N2;
    e = pass(N1, in_pair, OUT_COMPLEX, -1, N2, q, k, p->ws1, Nu * Wz, N * Wz, (int)Wz, 1, N2, 1, N2, 1, 1.0f);
    if (e != hipSuccess) goto fail;
    mark();
    // frequency w1 + N1 w2 goes to row w1 N2 + w2 (contiguous per block, see CgArgs)
    e = pass(N2, IN_COMPLEX, OUT_COMPLEX, -1, N1, p->ws1, nullptr, p->ws2, N * Wz, N * Wz, (int)Wz, N2, 1, N2, 1, 0,
             1.0f);
    if (e != hipSuccess) goto fail;
    mark();
    ca.Z = p->ws2;
    ca.W = p->ws1;
    ca.trash = p->ws1 + p->B * N * K * p->Cp;
    e = mix ? launch_mix(p->L, ca, s) : launch_cg(p->L, ca, p->force_generic, s);
    if (e != hipSuccess) goto fail;
    mark();
    e = pass(N2, IN_COMPLEX, OUT_COMPLEX, 1, N1, p->ws1, nullptr, p->ws2, N * Ww, N * Ww, (int)Ww, N2, 1, N2, 1, 1,
             1.0f);
    if (e != hipSuccess) goto fail;
    mark();
    e = pass(N1, IN_COMPLEX, out_split, 1, N2, p->ws2, nullptr, out, N * Ww, Nu * K * p->C, (int)Ww, 1, N2, 1, N2, 0,
             inv_n);
    if (e != hipSuccess) goto fail;
    mark();
  }
  return CGCONV_OK;
fail:
  set_error("kernel launch failed: %s", hipGetErrorString(e));
  return CGCONV_ERR_HIP;
}

// Inter-channel convolution with the per-degree reduction: the unfused
// forward passes over the C input channels, the inter-channel stage (Z ->
// packed output spectra of H*mo channels), the unfused inverse passes over
// the output channels.  The output spectra (B*N*K*H*mo/2 complex) fit in a
// workspace sized for C >= H*mo channels.
int run_interchannel(cgconv_plan* p, int heads, int mo, const float* q, const float* k, const float* wt, float* out,
                     hipStream_t s) {
  const int K = p->K;
  const int Co = heads * mo, Cpo = Co / 2;
  const long long Wz = (long long)K * p->C, Wo = (long long)K * Cpo;
  const long long N = p->N, Nu = p->Nu;
  const int in_pair = IN_PAIR_F32 + (p->linear ? 3 : 0);
  auto pass = [&](int R, int inm, int outm, int dir, int groups, const void* in0, const void* in1, void* o,
                  long long ib, long long ob, int W, int gs_in, int es_in, int gs_out, int fs_out, int inter,
                  float scale, bool output_side) {
    PassDesc d;
    d.R = R;
    d.in_mode = inm;
    d.out_mode = outm;
    d.dir = dir;
    d.groups = groups;
    d.batch = (int)p->B;
    d.a = base_args(p);
    if (output_side) {  // the inverse passes carry the H*mo output channels
      d.a.C = Co;
      d.a.Cp = Cpo;
      d.a.KC = K * Co;
    }
    d.a.in0 = in0;
    d.a.in1 = in1;
    d.a.out = o;
    d.a.in_bstride = ib;
    d.a.out_bstride = ob;
    d.a.W = W;
    d.a.gs_in = gs_in;
    d.a.es_in = es_in;
    d.a.gs_out = gs_out;
    d.a.fs_out = fs_out;
    d.a.tw_stride = (int)(p->N / R);
    d.a.inter = inter;
    d.a.scale = scale;
    return launch_fft_pass(d, s);
  };
  hipEvent_t* ev = nullptr;
  if (p->timing_calls < p->timing_max && (p->timing_kind < 0 || p->timing_kind == kKindInter)) {
    p->timing_kind = kKindInter;
    ev = &p->events[(size_t)p->timing_calls * kMaxEvents];
    ++p->timing_calls;
  }
  int stage = 0;
  auto mark = [&]() {
    if (ev) (void)hipEventRecord(ev[stage], s);
    ++stage;
  };
  InterArgs ia;
  ia.wt = wt;
  ia.N = N;
  ia.F = (int)(N / 2 + 1);
  ia.B = (int)p->B;
  ia.C = (int)p->C;
  ia.H = heads;
  ia.m = (int)(p->C / heads);
  ia.mo = mo;
  ia.Cpo = Cpo;
  const float inv_n = 1.0f / (float)N;
  hipError_t e;
  mark();
  if (p->N1 == 0) {
    if ((e = pass((int)N, in_pair, OUT_COMPLEX, -1, 1, q, k, p->ws1, Nu * Wz, N * Wz, (int)Wz, 0, 1, 0, 1, 0, 1.0f,
                  false)) != hipSuccess)
      goto fail;
    mark();
    ia.Z = p->ws1;
    ia.W = p->ws2;
    ia.n1_log2 = ilog2(N);
    ia.n2_log2 = 0;
    if ((e = launch_inter(p->L, ia, s)) != hipSuccess) goto fail;
    mark();
    if ((e = pass((int)N, IN_COMPLEX, OUT_SPLIT_F32, 1, 1, p->ws2, nullptr, out, N * Wo, Nu * K * Co, (int)Wo, 0, 1,
                  0, 1, 0, inv_n, true)) != hipSuccess)
      goto fail;
    mark();
  } else {
    const int N1 = (int)p->N1, N2 = (int)p->N2;
    if ((e = pass(N1, in_pair, OUT_COMPLEX, -1, N2, q, k, p->ws1, Nu * Wz, N * Wz, (int)Wz, 1, N2, 1, N2, 1, 1.0f,
                  false)) != hipSuccess)
      goto fail;
    mark();
    if ((e = pass(N2, IN_COMPLEX, OUT_COMPLEX, -1, N1, p->ws1, nullptr, p->ws2, N * Wz, N * Wz, (int)Wz, N2, 1, N2, 1,
                  0, 1.0f, false)) != hipSuccess)
      goto fail;
    mark();
    ia.Z = p->ws2;
    ia.W = p->ws1;
    ia.n1_log2 = ilog2(N1);
    ia.n2_log2 = ilog2(N2);
    if ((e = launch_inter(p->L, ia, s)) != hipSuccess) goto fail;
    mark();
    if ((e = pass(N2, IN_COMPLEX, OUT_COMPLEX, 1, N1, p->ws1, nullptr, p->ws2, N * Wo, N * Wo, (int)Wo, N2, 1, N2, 1,
                  1, 1.0f, true)) != hipSuccess)
      goto fail;
    mark();
    if ((e = pass(N1, IN_COMPLEX, OUT_SPLIT_F32, 1, N2, p->ws2, nullptr, out, N * Wo, Nu * K * Co, (int)Wo, 1, N2, 1,
                  N2, 0, inv_n, true)) != hipSuccess)
      goto fail;
    mark();
  }
  return CGCONV_OK;
fail:
  set_error("kernel launch failed: %s", hipGetErrorString(e));
  return CGCONV_ERR_HIP;
}

int check_plan_args(cgconv_plan* p, const void* q, const void* k, const void* out) {
  if (!p) {
    set_error("plan is NULL");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (!q || !k || !out) {
    set_error("q, k and out must be non-NULL device pointers");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (!aligned16(q) || !aligned16(k) || !aligned16(out)) {
    set_error("q, k and out must be 16-byte aligned");
    return CGCONV_ERR_ALIGNMENT;
  }
  if (out == q || out == k) {
    set_error("out must not alias q or k");
    return CGCONV_ERR_INVALID_ARG;
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != p->device) {
    set_error("the plan's device (%d) is not current (%d)", p->device, cur);
    return CGCONV_ERR_INVALID_ARG;
  }
  return CGCONV_OK;
}

// Backward scales.  The real-basis coefficients obey, path by path,
//   R^(J l2 l1)[m1, M, m2] = (-1)^l2 sqrt((2 l1 + 1) / (2 J + 1)) R^(l1 l2 J)[M, m1, m2],
// so each gradient is the forward convolution of the output gradient g
// with the other operand time-reversed (token DFT) or as is (graph basis),
// under per-degree scales:
//   dq = s_o * conv(s_a * g, s_b * k'):  s_a = sqrt(2l+1), s_b = (-1)^l, s_o = 1/sqrt(2l+1)
//   dk = s_o * conv(s_a * g, q'):        s_a = (-1)^l sqrt(2l+1), s_b = 1, s_o = (-1)^l/sqrt(2l+1)
// Table [dq: s_a, s_b, s_o][dk: s_a, s_b, s_o], K floats each.
hipError_t upload_backward_scales(cgconv_plan* p) {
  const int K = p->K;
  std::vector<float> bs(6 * (size_t)K);
  for (int l = 0; l <= p->L; ++l) {
    const double r = std::sqrt(2.0 * l + 1.0), sg = (l & 1) ? -1.0 : 1.0;
    for (int c = l * l; c < (l + 1) * (l + 1); ++c) {
      bs[c] = (float)r;
      bs[K + c] = (float)sg;
      bs[2 * K + c] = (float)(1.0 / r);
      bs[3 * K + c] = (float)(sg * r);
      bs[4 * K + c] = 1.0f;
      bs[5 * K + c] = (float)(sg / r);
    }
  }
  return upload(&p->d_bscale, bs);
}

// gating partials: ceil(Nu / kGateChunk) chunks per batch element
hipError_t alloc_gate_workspace(cgconv_plan* p) {
  const size_t chunks = (size_t)((p->Nu + kGateChunk - 1) / kGateChunk);
  const size_t np = (size_t)p->B * chunks * (p->L + 1) * p->C, nf = (size_t)p->B * (p->L + 1) * p->C;
  hipError_t e;
  if ((e = hipMalloc(&p->d_gpart, np * sizeof(float2))) != hipSuccess) return e;
  if ((e = hipMalloc(&p->d_gfin, nf * sizeof(float2))) != hipSuccess) return e;
  const size_t nh = (size_t)p->B * p->Nu * (p->L + 1) * p->C;
  if ((e = hipMalloc(&p->d_gh, nh * sizeof(float))) != hipSuccess) return e;
  if ((e = hipMalloc(&p->d_gS, nf * sizeof(float))) != hipSuccess) return e;
  p->ws_bytes += (np + nf) * sizeof(float2) + (nh + nf) * sizeof(float);
  return hipSuccess;
}

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// distinct complex products q[l1,m1] * k[l2,m2] among the contraction terms
int64_t distinct_products(const std::vector<Term>& terms, int K) {
  std::vector<char> seen((size_t)K * K, 0);
  int64_t n = 0;
  for (const Term& t : terms) {
    char& f = seen[(size_t)comp(t.l1, t.m1) * K + comp(t.l2, t.m2)];
    n += f == 0;
    f = 1;
  }
  return n;
}

// the token-DFT entry points: everything but a graph plan
int check_forward_args(cgconv_plan* p, const void* q, const void* k, const void* out) {
  const int st = check_plan_args(p, q, k, out);
  if (st == CGCONV_OK && p->graph) {
    set_error("a graph plan takes cgconv_forward_graph (or cgconv_gate_value)");
    return CGCONV_ERR_INVALID_ARG;
  }
  return st;
}

}  // namespace

extern "C" {

const char* cgconv_last_error(void) { return g_last_error.c_str(); }

cgconv_plan_t cgconv_plan_create(int64_t batch, int64_t N, int32_t L_max, int64_t C) {
  return cgconv_plan_create_boundary(batch, N, L_max, C, CGCONV_BOUNDARY_CYCLIC);
}

cgconv_plan_t cgconv_plan_create_boundary(int64_t batch, int64_t N_tokens, int32_t L_max, int64_t C,
                                          int32_t boundary) {
  g_last_error.clear();
  if (boundary != CGCONV_BOUNDARY_CYCLIC && boundary != CGCONV_BOUNDARY_LINEAR) {
    set_error("invalid boundary=%d", boundary);
    return nullptr;
  }
  const bool linear = boundary == CGCONV_BOUNDARY_LINEAR;
  if (batch < 1 || C < 1 || N_tokens < (linear ? 1 : 2)) {
    set_error("invalid sizes: batch=%lld N=%lld C=%lld (need batch>=1, N>=%d, C>=1)", (long long)batch,
              (long long)N_tokens, (long long)C, linear ? 1 : 2);
    return nullptr;
  }
  if (L_max < 0) {
    set_error("invalid L_max=%d", L_max);
    return nullptr;
  }
  // DFT length: N itself (cyclic), or the smallest power of two >= 2N - 1 so
  // that no term of the zero-padded sum wraps around (linear)
  int64_t N = N_tokens;
  if (linear) {
    if (N_tokens > CGCONV_NMAX / 2) {
      set_error("unsupported N=%lld: the linear boundary needs N <= %d", (long long)N_tokens, CGCONV_NMAX / 2);
      return nullptr;
    }
    N = 2;
    while (N < 2 * N_tokens - 1) N *= 2;
  } else if (!is_pow2(N) || N > CGCONV_NMAX) {
    set_error("unsupported N=%lld: need a power of two <= %d", (long long)N, CGCONV_NMAX);
    return nullptr;
  }
  if (L_max > CGCONV_LMAX) {
    set_error("unsupported L_max=%d: at most %d", L_max, CGCONV_LMAX);
    return nullptr;
  }
  const int K = (L_max + 1) * (L_max + 1);
  const int64_t Cp = (C + 1) / 2;
  // sizes must keep every element index and grid dimension in range
  const long double elems = (long double)batch * N * K * C;
  if (elems > 4.0e9L || batch > 65535) {
    set_error("problem too large: batch*N*K*C=%.3Le (max 4e9), batch=%lld (max 65535)", elems, (long long)batch);
    return nullptr;
  }
  cgconv_plan* p = new (std::nothrow) cgconv_plan;
  if (!p) {
    set_error("host allocation failed");
    return nullptr;
  }
  p->B = batch;
  p->N = N;
  p->Nu = N_tokens;
  p->linear = linear;
  p->C = C;
  p->Cp = Cp;
  p->L = L_max;
  p->K = K;
  if (const char* env = std::getenv("CGCONV_FORCE_GENERIC")) p->force_generic = env[0] == '1';
  const char* unfused = std::getenv("CGCONV_UNFUSED");
  // the fused kernel addresses one batch element's spectra with 32-bit byte offsets
  const bool fits32 = (long double)N * K * C * 8 < 4294967296.0L;
  if (N >= 512 && N <= 32768 && L_max <= kFusedLmax && fits32 && !(unfused && unfused[0] == '1') &&
      !p->force_generic) {
    p->fused = true;
    p->N2 = 64;
    p->N1 = N / 64;
  } else if (N > 256) {
    const int lg = ilog2(N);
    p->N1 = int64_t(1) << ((lg + 1) / 2);
    p->N2 = N / p->N1;
  }
  p->n_stages = (p->N1 && !p->fused) ? 5 : 3;
  p->n_stages_mix = p->N1 ? 5 : 3;
  // DFT length <= 256: the one-block kernel, with the smallest channel group
  // (a power of two, 2 .. 16) that gives a block at least 256 lanes (two per
  // point), within the thread and LDS limits
  const char* no_small = std::getenv("CGCONV_NO_SMALL");
  if (N <= kSmallMaxNf && L_max <= kSmallLmax && !p->force_generic && !(no_small && no_small[0] == '1')) {
    const int64_t per_ch = 2 * (N / 2 + 1);  // lanes per channel
    const int max_threads = small_max_threads(L_max);
    int cc = 2;
    while (2 * cc <= 16 && cc < 2 * Cp && per_ch * cc < 256 && per_ch * 2 * cc <= max_threads &&
           small_lds_bytes(N, K, 2 * cc) <= kSmallMaxLds)
      cc *= 2;
    const int64_t threads = (per_ch * cc + 63) / 64 * 64;
    // a block reads cc of every C channels of a row: with fewer than a
    // quarter, the loads touch so many more cache lines than they use that
    // the three kernels, each reading whole rows, are faster (n-body size:
    // one block 34 us, three kernels 28 us; tiny 10 against 14 us, molecule
    // size 26 against 27 us)
    if (threads <= max_threads && small_lds_bytes(N, K, cc) <= kSmallMaxLds && 4 * cc >= C) {
      p->small = true;
      p->small_cc = cc;
      p->small_threads = (int)threads;
    }
  }
  hipError_t e = hipGetDevice(&p->device);
  if (e != hipSuccess) {
    set_error("hipGetDevice failed: %s", hipGetErrorString(e));
    delete p;
    return nullptr;
  }
  if (p->small && small_lds_bytes(N, K, p->small_cc) > 64 * 1024 &&
      (e = prepare_small(L_max, (int)small_lds_bytes(N, K, p->small_cc))) != hipSuccess) {
    set_error("hipFuncSetAttribute failed: %s", hipGetErrorString(e));
    delete p;
    return nullptr;
  }
  // twiddles exp(-2 pi i j / N), computed in double and rounded once
  std::vector<float2> tw(N);
  for (int64_t j = 0; j < N; ++j) {
    const double ang = -2.0 * M_PI * (double)j / (double)N;
    tw[j] = make_float2((float)std::cos(ang), (float)std::sin(ang));
  }
  // table for the generic contraction kernel, grouped by complex-basis output
  std::vector<Term> terms = contraction_terms(L_max);
  std::vector<int> offs(K + 1, 0);
  std::vector<uint32_t> tkey(terms.size());
  std::vector<float> tcoef(terms.size());
  for (const Term& t : terms) offs[comp(t.J, t.M) + 1]++;
  for (int o = 0; o < K; ++o) offs[o + 1] += offs[o];
  {
    std::vector<int> fill(offs.begin(), offs.end() - 1);
    for (const Term& t : terms) {
      const int pos = fill[comp(t.J, t.M)]++;
      tkey[pos] = (uint32_t)comp(t.l1, t.m1) | ((uint32_t)comp(t.l2, t.m2) << 8) | ((t.imag ? 1u : 0u) << 16);
      tcoef[pos] = (float)t.coef;
    }
  }
  p->nnz = (int64_t)terms.size();
  if (!evaluated_table(L_max, terms, p->rtable)) {
    set_error("internal error: the contraction terms do not expand to a real tensor");
    delete p;
    return nullptr;
  }
  p->products = distinct_products(terms, K);
  p->paths = n_paths(L_max);
  // each workspace holds a [B][N][K][C] float2 array, followed by a trash area
  // that absorbs the masked stores of the CG stage (K*Cp float2, at least 256)
  const size_t trash = std::max<size_t>((size_t)K * Cp, 256);
  const size_t ws = ((size_t)batch * N * K * C + trash) * sizeof(float2);
  p->ws_bytes = 2 * ws;
  if (const char* env = std::getenv("CGCONV_TEST_FAIL_ALLOC"); env && env[0] == '1') {
    set_error("workspace allocation of %zu bytes failed (forced by CGCONV_TEST_FAIL_ALLOC)", p->ws_bytes);
    delete p;
    return nullptr;
  }
  if ((e = hipMalloc(&p->ws1, ws)) != hipSuccess || (e = hipMalloc(&p->ws2, ws)) != hipSuccess) {
    set_error("workspace allocation of %zu bytes failed: %s", p->ws_bytes, hipGetErrorString(e));
    (void)hipGetLastError();
    free_plan(p);
    return nullptr;
  }
  if ((e = upload(&p->tw, tw)) != hipSuccess || (e = upload(&p->d_offs, offs)) != hipSuccess ||
      (e = upload(&p->d_tkey, tkey)) != hipSuccess || (e = upload(&p->d_tcoef, tcoef)) != hipSuccess) {
    set_error("table upload failed: %s", hipGetErrorString(e));
    free_plan(p);
    return nullptr;
  }
  if ((e = alloc_gate_workspace(p)) != hipSuccess) {
    set_error("gating workspace allocation failed: %s", hipGetErrorString(e));
    (void)hipGetLastError();
    free_plan(p);
    return nullptr;
  }
  if ((e = upload_backward_scales(p)) != hipSuccess) {
    set_error("backward scale upload failed: %s", hipGetErrorString(e));
    (void)hipGetLastError();
    free_plan(p);
    return nullptr;
  }
  if (L_max <= kMixLmax && C <= kMixCmax) {
    // prepared channel-mixing weights, 2048 bf16 per path
    if ((e = hipMalloc(&p->d_wmix, (size_t)p->paths * 2048 * sizeof(uint16_t))) != hipSuccess) {
      set_error("mixing-weight allocation failed: %s", hipGetErrorString(e));
      (void)hipGetLastError();
      free_plan(p);
      return nullptr;
    }
    p->ws_bytes += (size_t)p->paths * 2048 * sizeof(uint16_t);
  }
  return p;
}

void cgconv_plan_destroy(cgconv_plan_t plan) { free_plan(plan); }

cgconv_plan_t cgconv_plan_create_graph(int64_t batch, int64_t N, int32_t L_max, int64_t C) {
  g_last_error.clear();
  if (batch < 1 || C < 1 || N < 1 || batch > 65535) {
    set_error("invalid sizes: batch=%lld N=%lld C=%lld (need 1 <= batch <= 65535, N>=1, C>=1)", (long long)batch,
              (long long)N, (long long)C);
    return nullptr;
  }
  if (L_max < 0 || L_max > CGCONV_LMAX) {
    set_error("unsupported L_max=%d: 0..%d", L_max, CGCONV_LMAX);
    return nullptr;
  }
  if (N > CGCONV_GRAPH_NMAX) {
    set_error("unsupported N=%lld: a graph plan holds N x N bases, N <= %d", (long long)N, CGCONV_GRAPH_NMAX);
    return nullptr;
  }
  cgconv_plan* p = new (std::nothrow) cgconv_plan;
  if (!p) {
    set_error("host allocation failed");
    return nullptr;
  }
  const int K = (L_max + 1) * (L_max + 1);
  p->graph = true;
  p->B = batch;
  p->N = N;
  p->Nu = N;
  p->C = C;
  p->Cp = (C + 1) / 2;
  p->L = L_max;
  p->K = K;
  p->paths = n_paths(L_max);
  {
    const std::vector<Term> terms = contraction_terms(L_max);
    p->nnz = (int64_t)terms.size();
    p->products = distinct_products(terms, K);
  }
  p->rtable = real_table(L_max);  // the per-frequency product is the generated real-basis body
  p->Kp = round_up(N, 32);
  p->Mp = round_up(N, 128);
  p->KCp = round_up((int64_t)K * C, 128);
  hipError_t e = hipGetDevice(&p->device);
  if (e != hipSuccess) {
    set_error("hipGetDevice failed: %s", hipGetErrorString(e));
    delete p;
    return nullptr;
  }
  // sub-buffers of one allocation, each 256-byte aligned
  const size_t a_elems = (size_t)batch * p->Mp * p->Kp, bf_elems = (size_t)batch * 2 * p->KCp * p->Kp,
               bi_elems = (size_t)batch * p->KCp * p->Kp;
  const size_t spec_elems = (size_t)batch * N * 2 * p->KCp, uhat_elems = (size_t)batch * N * K * C;
  const size_t sizes[] = {a_elems * 2, a_elems * 2, a_elems * 2, a_elems * 2, bf_elems * 2, bf_elems * 2,
                          bi_elems * 2, bi_elems * 2, spec_elems * 4, uhat_elems * 4};
  size_t offs[10], total = 0;
  for (int i = 0; i < 10; ++i) {
    offs[i] = total;
    total += (sizes[i] + 255) / 256 * 256;
  }
  if ((e = hipMalloc(&p->g_block, total)) != hipSuccess) {
    set_error("graph workspace allocation of %zu bytes failed: %s", total, hipGetErrorString(e));
    (void)hipGetLastError();
    delete p;
    return nullptr;
  }
  char* base = static_cast<char*>(p->g_block);
  p->ga_fh = reinterpret_cast<uint16_t*>(base + offs[0]);
  p->ga_fl = reinterpret_cast<uint16_t*>(base + offs[1]);
  p->ga_ih = reinterpret_cast<uint16_t*>(base + offs[2]);
  p->ga_il = reinterpret_cast<uint16_t*>(base + offs[3]);
  p->gb_fh = reinterpret_cast<uint16_t*>(base + offs[4]);
  p->gb_fl = reinterpret_cast<uint16_t*>(base + offs[5]);
  p->gb_ih = reinterpret_cast<uint16_t*>(base + offs[6]);
  p->gb_il = reinterpret_cast<uint16_t*>(base + offs[7]);
  p->g_spec = reinterpret_cast<float*>(base + offs[8]);
  p->g_uhat = reinterpret_cast<float*>(base + offs[9]);
  p->ws_bytes = total;
  if ((e = alloc_gate_workspace(p)) != hipSuccess || (e = upload_backward_scales(p)) != hipSuccess) {
    set_error("graph plan set-up failed: %s", hipGetErrorString(e));
    (void)hipGetLastError();
    free_plan(p);
    return nullptr;
  }
  return p;
}

}  // extern "C"

namespace {

// One graph pipeline: out = U R:((U^T x1) (x) (U^T x2)), with per-component
// scales of the product when `scales` is set; split_u = false reuses the
// split bases of the previous pipeline on this plan.
int run_graph(cgconv_plan* p, const float* U, const float* x1, const float* x2, float* out, const float* scales,
              bool split_u, hipStream_t stream) {
  hipEvent_t* ev = nullptr;
  if (p->timing_calls < p->timing_max && (p->timing_kind < 0 || p->timing_kind == kKindGraph)) {
    p->timing_kind = kKindGraph;
    ev = &p->events[(size_t)p->timing_calls * kMaxEvents];
    ++p->timing_calls;
  }
  int stage = 0;
  auto mark = [&]() {
    if (ev) (void)hipEventRecord(ev[stage], stream);
    ++stage;
  };
  const int B = (int)p->B, n = (int)p->N, KC = p->K * (int)p->C;
  const int Kp = (int)p->Kp, Mp = (int)p->Mp, KCp = (int)p->KCp;
  auto split = [&](const float* src, long long src_bs, int ld, int rows, int cols, uint16_t* hi, uint16_t* lo,
                   long long dst_bs, int dst_rows, int row0, int dst_rt, uint16_t* hi_p = nullptr,
                   uint16_t* lo_p = nullptr) {
    GftSplitArgs a;
    a.src = src;
    a.src_bs = src_bs;
    a.ld = ld;
    a.src_rows = rows;
    a.src_cols = cols;
    a.hi = hi;
    a.lo = lo;
    a.hi_p = hi_p;
    a.lo_p = lo_p;
    a.dst_bs = dst_bs;
    a.dst_rows = dst_rows;
    a.dst_cols = Kp;
    a.row0 = row0;
    a.dst_rt = dst_rt;
    return launch_gft_split(a, B, stream);
  };
  auto gemm = [&](const uint16_t* ah, const uint16_t* al, const uint16_t* bh, const uint16_t* bl, long long b_bs,
                  float* c, long long c_bs, int ldc, int N_, int Np) {
    GftGemmArgs g;
    g.ah = ah;
    g.al = al;
    g.bh = bh;
    g.bl = bl;
    g.a_bs = (long long)Mp * Kp;
    g.b_bs = b_bs;
    g.c = c;
    g.c_bs = c_bs;
    g.ldc = ldc;
    g.M = n;
    g.N = N_;
    g.Kp = Kp;
    return launch_gft_gemm(g, Mp, Np, B, stream);
  };
  const long long nn = (long long)n * n, xbs = (long long)n * KC;
  hipError_t e;
  mark();
  // A operands: U^T (rows = graph frequencies) and U (rows = nodes), k = the other index
  if (split_u) {  // U^T and U from one read of U
    if ((e = split(U, nn, n, n, n, p->ga_fh, p->ga_fl, (long long)Mp * Kp, Mp, 0, Mp / 128, p->ga_ih, p->ga_il)) !=
        hipSuccess)
      goto fail;
  }
  mark();
  // B operand of the forward transform: [q | k] transposed, q in rows 0..KC-1, k from row KCp
  if ((e = split(x1, xbs, KC, n, KC, p->gb_fh, p->gb_fl, 2LL * KCp * Kp, KCp, 0, 2 * KCp / 128)) != hipSuccess)
    goto fail;
  if ((e = split(x2, xbs, KC, n, KC, p->gb_fh, p->gb_fl, 2LL * KCp * Kp, KCp, KCp, 2 * KCp / 128)) != hipSuccess)
    goto fail;
  mark();
  // [q_hat | k_hat] = U^T [q | k]
  if ((e = gemm(p->ga_fh, p->ga_fl, p->gb_fh, p->gb_fl, 2LL * KCp * Kp, p->g_spec, (long long)n * 2 * KCp, 2 * KCp,
                2 * KCp, 2 * KCp)) != hipSuccess)
    goto fail;
  mark();
  {
    GftProductArgs a;
    a.spec = p->g_spec;
    a.spec_bs = (long long)n * 2 * KCp;
    a.ld = 2 * KCp;
    a.kb_off = KCp;
    a.out = p->g_uhat;
    a.out_bs = xbs;
    a.B = B;
    a.n = n;
    a.C = (int)p->C;
    a.scales = scales;
    if ((e = launch_product(p->L, a, stream)) != hipSuccess) goto fail;
  }
  mark();
  if ((e = split(p->g_uhat, xbs, KC, n, KC, p->gb_ih, p->gb_il, (long long)KCp * Kp, KCp, 0, KCp / 128)) !=
      hipSuccess)
    goto fail;
  mark();
  // u = U u_hat, written straight into out ([B][n][K][C] = [B][n][KC])
  if ((e = gemm(p->ga_ih, p->ga_il, p->gb_ih, p->gb_il, (long long)KCp * Kp, out, xbs, KC, KC, KCp)) != hipSuccess)
    goto fail;
  mark();
  return CGCONV_OK;
fail:
  set_error("kernel launch failed: %s", hipGetErrorString(e));
  return CGCONV_ERR_HIP;
}

}  // namespace

extern "C" {

int cgconv_forward_graph(cgconv_plan_t plan, const float* U, const float* q, const float* k, float* out,
                         hipStream_t stream) {
  const int st = check_plan_args(plan, q, k, out);
  if (st != CGCONV_OK) return st;
  if (!plan->graph) {
    set_error("cgconv_forward_graph needs a plan from cgconv_plan_create_graph");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (!U) {
    set_error("U must be a non-NULL device pointer");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (!aligned16(U)) {
    set_error("U must be 16-byte aligned");
    return CGCONV_ERR_ALIGNMENT;
  }
  if (out == U) {
    set_error("out must not alias U");
    return CGCONV_ERR_INVALID_ARG;
  }
  return run_graph(plan, U, q, k, out, nullptr, true, stream);
}

int cgconv_backward_graph(cgconv_plan_t plan, const float* U, const float* q, const float* k, const float* grad_out,
                          float* grad_q, float* grad_k, hipStream_t stream) {
  if (!plan || !plan->graph) {
    set_error("cgconv_backward_graph needs a plan from cgconv_plan_create_graph");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (!U || !q || !k || !grad_out || (!grad_q && !grad_k)) {
    set_error("U, q, k and grad_out must be non-NULL, and at least one of grad_q, grad_k");
    return CGCONV_ERR_INVALID_ARG;
  }
  const void* ptrs[] = {U, q, k, grad_out, grad_q, grad_k};
  for (const void* ptr : ptrs) {
    if (ptr && !aligned16(ptr)) {
      set_error("U, q, k, grad_out, grad_q and grad_k must be 16-byte aligned");
      return CGCONV_ERR_ALIGNMENT;
    }
  }
  for (const float* g : {grad_q, grad_k}) {
    if (g && (g == U || g == q || g == k || g == grad_out)) {
      set_error("grad_q and grad_k must not alias U, q, k or grad_out");
      return CGCONV_ERR_INVALID_ARG;
    }
  }
  if (grad_q && grad_q == grad_k) {
    set_error("grad_q and grad_k must be distinct");
    return CGCONV_ERR_INVALID_ARG;
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != plan->device) {
    set_error("the plan's device (%d) is not current (%d)", plan->device, cur);
    return CGCONV_ERR_INVALID_ARG;
  }
  const int K = plan->K;
  bool split_u = true;
  if (grad_q) {
    const int st = run_graph(plan, U, grad_out, k, grad_q, plan->d_bscale, true, stream);
    if (st != CGCONV_OK) return st;
    split_u = false;
  }
  if (grad_k) return run_graph(plan, U, grad_out, q, grad_k, plan->d_bscale + 3 * K, split_u, stream);
  return CGCONV_OK;
}

int cgconv_plan_info(cgconv_plan_t plan, int64_t* n_paths_out, int64_t* nnz, size_t* workspace_bytes) {
  if (!plan) {
    set_error("plan is NULL");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (n_paths_out) *n_paths_out = plan->paths;
  if (nnz) *nnz = (int64_t)plan->rtable.size();
  if (workspace_bytes) *workspace_bytes = plan->ws_bytes;
  return CGCONV_OK;
}

int cgconv_plan_contraction_info(cgconv_plan_t plan, int64_t* nnz_complex, int64_t* n_products) {
  if (!plan) {
    set_error("plan is NULL");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (nnz_complex) *nnz_complex = plan->nnz;
  if (n_products) *n_products = plan->products;
  return CGCONV_OK;
}

int64_t cgconv_plan_export_table(cgconv_plan_t plan, int32_t* l1m1l2m2JM, double* coef, int64_t cap) {
  if (!plan) {
    set_error("plan is NULL");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (cap < 0 || (cap > 0 && (!l1m1l2m2JM || !coef))) {
    set_error("invalid output buffers");
    return CGCONV_ERR_INVALID_ARG;
  }
  const std::vector<RealEntry>& t = plan->rtable;
  for (int64_t e = 0; e < (int64_t)t.size() && e < cap; ++e) {
    const RealEntry& r = t[e];
    const int32_t v[6] = {r.l1, r.m1, r.l2, r.m2, r.J, r.M};
    std::memcpy(l1m1l2m2JM + 6 * e, v, sizeof v);
    coef[e] = r.coef;
  }
  return (int64_t)t.size();
}

int cgconv_plan_enable_timing(cgconv_plan_t plan, int32_t max_calls) {
  if (!plan || max_calls < 0) {
    set_error("plan is NULL or max_calls < 0");
    return CGCONV_ERR_INVALID_ARG;
  }
  for (hipEvent_t ev : plan->events) (void)hipEventDestroy(ev);
  plan->events.clear();
  plan->timing_max = 0;
  plan->timing_calls = 0;
  plan->timing_kind = -1;
  const size_t n = (size_t)max_calls * kMaxEvents;
  plan->events.reserve(n);
  for (size_t i = 0; i < n; ++i) {
    hipEvent_t ev;
    const hipError_t e = hipEventCreate(&ev);
    if (e != hipSuccess) {
      set_error("hipEventCreate failed: %s", hipGetErrorString(e));
      for (hipEvent_t x : plan->events) (void)hipEventDestroy(x);
      plan->events.clear();
      return CGCONV_ERR_HIP;
    }
    plan->events.push_back(ev);
  }
  plan->timing_max = max_calls;
  return CGCONV_OK;
}

int cgconv_plan_stage_times(cgconv_plan_t plan, double* ms, int32_t cap, int32_t* n_stages, int32_t* n_calls) {
  if (!plan || (cap > 0 && !ms)) {
    set_error("plan is NULL or ms is NULL");
    return CGCONV_ERR_INVALID_ARG;
  }
  const int ns = plan->timing_kind == 1 || plan->timing_kind == kKindInter ? plan->n_stages_mix
                 : plan->timing_kind == kKindSmall ? 1
                 : plan->timing_kind == kKindGate  ? 3
                 : plan->timing_kind == kKindGateBwd ? 4
                 : plan->timing_kind == kKindGraph ? 6
                                                   : plan->n_stages;
  if (n_stages) *n_stages = ns;
  if (n_calls) *n_calls = plan->timing_calls;
  for (int st = 0; st < cap && st < ns; ++st) ms[st] = 0.0;
  for (int c = 0; c < plan->timing_calls; ++c) {
    hipEvent_t* ev = &plan->events[(size_t)c * kMaxEvents];
    hipError_t e = hipEventSynchronize(ev[ns]);
    if (e != hipSuccess) {
      set_error("hipEventSynchronize failed: %s", hipGetErrorString(e));
      return CGCONV_ERR_HIP;
    }
    for (int st = 0; st < cap && st < ns; ++st) {
      float t = 0.f;
      e = hipEventElapsedTime(&t, ev[st], ev[st + 1]);
      if (e != hipSuccess) {
        set_error("hipEventElapsedTime failed: %s", hipGetErrorString(e));
        return CGCONV_ERR_HIP;
      }
      ms[st] += t;
    }
  }
  return CGCONV_OK;
}

const char* cgconv_plan_stage_name(cgconv_plan_t plan, int32_t stage) {
  if (!plan || stage < 0) return "";
  if (plan->timing_kind == 1) {
    if (stage >= plan->n_stages_mix) return "";
    return plan->N1 ? kStagesM2[stage] : kStagesM1[stage];
  }
  if (plan->timing_kind == kKindSmall) return stage < 1 ? kStagesS[stage] : "";
  if (plan->timing_kind == kKindGate) return stage < 3 ? kStagesG[stage] : "";
  if (plan->timing_kind == kKindGateBwd) return stage < 4 ? kStagesGB[stage] : "";
  if (plan->timing_kind == kKindGraph) return stage < 6 ? kStagesGft[stage] : "";
  if (plan->timing_kind == kKindInter) {
    if (stage >= plan->n_stages_mix) return "";
    return plan->N1 ? kStagesI2[stage] : kStagesI1[stage];
  }
  if (stage >= plan->n_stages) return "";
  if (plan->fused) return kStagesF[stage];
  return plan->N1 ? kStages2[stage] : kStages1[stage];
}

int cgconv_forward(cgconv_plan_t plan, const float* q, const float* k, float* out, hipStream_t stream) {
  const int st = check_forward_args(plan, q, k, out);
  if (st != CGCONV_OK) return st;
  return run_forward(plan, q, k, out, false, stream);
}

int cgconv_forward_bf16(cgconv_plan_t plan, const uint16_t* q, const uint16_t* k, uint16_t* out,
                        hipStream_t stream) {
  const int st = check_forward_args(plan, q, k, out);
  if (st != CGCONV_OK) return st;
  return run_forward(plan, q, k, out, true, stream);
}

int cgconv_forward_mixed(cgconv_plan_t plan, const float* q, const float* k, const float* weights, float* out,
                         hipStream_t stream) {
  const int st = check_forward_args(plan, q, k, out);
  if (st != CGCONV_OK) return st;
  if (!weights) {
    set_error("weights must be a non-NULL device pointer");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (!aligned16(weights)) {
    set_error("weights must be 16-byte aligned");
    return CGCONV_ERR_ALIGNMENT;
  }
  if (!plan->d_wmix) {
    set_error("channel mixing needs L_max <= %d and C <= %d (plan: L_max=%d, C=%lld)", kMixLmax, kMixCmax, plan->L,
              (long long)plan->C);
    return CGCONV_ERR_UNSUPPORTED;
  }
  return run_forward(plan, q, k, out, false, stream, weights);
}

int cgconv_forward_interchannel(cgconv_plan_t plan, int32_t heads, int32_t m_out, const float* q, const float* k,
                                const float* weights, float* out, hipStream_t stream) {
  const int st = check_forward_args(plan, q, k, out);
  if (st != CGCONV_OK) return st;
  if (!weights) {
    set_error("weights must be a non-NULL device pointer");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (!aligned16(weights)) {
    set_error("weights must be 16-byte aligned");
    return CGCONV_ERR_ALIGNMENT;
  }
  if (weights == out) {
    set_error("out must not alias the weights");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (heads < 1 || plan->C % heads != 0 || m_out < 1) {
    set_error("invalid heads=%d or m_out=%d for C=%lld (heads must divide C, m_out >= 1)", heads, m_out,
              (long long)plan->C);
    return CGCONV_ERR_INVALID_ARG;
  }
  const int m = (int)(plan->C / heads);
  if (plan->L > kInterLmax || m > kInterMmax || m_out > m || (m_out & 1)) {
    set_error("unsupported inter-channel shape: needs L_max <= %d (plan: %d), m = C/heads <= %d (%d), m_out even and "
              "<= m (%d)",
              kInterLmax, plan->L, kInterMmax, m, m_out);
    return CGCONV_ERR_UNSUPPORTED;
  }
  return run_interchannel(plan, heads, m_out, q, k, weights, out, stream);
}

int cgconv_backward(cgconv_plan_t plan, const float* q, const float* k, const float* grad_out, float* grad_q,
                    float* grad_k, hipStream_t stream) {
  if (!plan) {
    set_error("plan is NULL");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (plan->graph) {
    set_error("a graph plan takes cgconv_forward_graph (or cgconv_gate_value)");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (!q || !k || !grad_out || (!grad_q && !grad_k)) {
    set_error("q, k and grad_out must be non-NULL, and at least one of grad_q, grad_k");
    return CGCONV_ERR_INVALID_ARG;
  }
  const void* ptrs[] = {q, k, grad_out, grad_q, grad_k};
  for (const void* ptr : ptrs) {
    if (ptr && !aligned16(ptr)) {
      set_error("q, k, grad_out, grad_q and grad_k must be 16-byte aligned");
      return CGCONV_ERR_ALIGNMENT;
    }
  }
  for (const float* g : {grad_q, grad_k}) {
    if (g && (g == q || g == k || g == grad_out)) {
      set_error("grad_q and grad_k must not alias q, k or grad_out");
      return CGCONV_ERR_INVALID_ARG;
    }
  }
  if (grad_q && grad_q == grad_k) {
    set_error("grad_q and grad_k must be distinct");
    return CGCONV_ERR_INVALID_ARG;
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != plan->device) {
    set_error("the plan's device (%d) is not current (%d)", plan->device, cur);
    return CGCONV_ERR_INVALID_ARG;
  }
  const int K = plan->K;
  if (grad_q) {
    const int st = run_forward(plan, grad_out, k, grad_q, false, stream, nullptr, plan->d_bscale);
    if (st != CGCONV_OK) return st;
  }
  if (grad_k) return run_forward(plan, grad_out, q, grad_k, false, stream, nullptr, plan->d_bscale + 3 * K);
  return CGCONV_OK;
}

int cgconv_gate_value(cgconv_plan_t plan, const float* u, const float* v, float* f, hipStream_t stream) {
  const int st = check_plan_args(plan, u, v, f);
  if (st != CGCONV_OK) return st;
  GateArgs a;
  a.u = u;
  a.v = v;
  a.f = f;
  a.part = plan->d_gpart;
  a.fin = plan->d_gfin;
  a.B = (int)plan->B;
  a.N = (int)plan->Nu;  // the softmax runs over the caller's tokens
  a.C = (int)plan->C;
  a.events = nullptr;
  if (plan->timing_calls < plan->timing_max && (plan->timing_kind < 0 || plan->timing_kind == kKindGate)) {
    plan->timing_kind = kKindGate;
    a.events = &plan->events[(size_t)plan->timing_calls * kMaxEvents];
    ++plan->timing_calls;
  }
  const hipError_t e = launch_gate(plan->L, a, stream);
  if (e != hipSuccess) {
    set_error("kernel launch failed: %s", hipGetErrorString(e));
    return CGCONV_ERR_HIP;
  }
  return CGCONV_OK;
}

int cgconv_gate_value_backward(cgconv_plan_t plan, const float* u, const float* v, const float* grad_f,
                               float* grad_u, float* grad_v, hipStream_t stream) {
  if (!plan) {
    set_error("plan is NULL");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (!u || !v || !grad_f || (!grad_u && !grad_v)) {
    set_error("u, v and grad_f must be non-NULL, and at least one of grad_u, grad_v");
    return CGCONV_ERR_INVALID_ARG;
  }
  const void* ptrs[] = {u, v, grad_f, grad_u, grad_v};
  for (const void* ptr : ptrs) {
    if (ptr && !aligned16(ptr)) {
      set_error("u, v, grad_f, grad_u and grad_v must be 16-byte aligned");
      return CGCONV_ERR_ALIGNMENT;
    }
  }
  for (const float* g : {grad_u, grad_v}) {
    if (g && (g == u || g == v || g == grad_f)) {
      set_error("grad_u and grad_v must not alias u, v or grad_f");
      return CGCONV_ERR_INVALID_ARG;
    }
  }
  if (grad_u && grad_u == grad_v) {
    set_error("grad_u and grad_v must be distinct");
    return CGCONV_ERR_INVALID_ARG;
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != plan->device) {
    set_error("the plan's device (%d) is not current (%d)", plan->device, cur);
    return CGCONV_ERR_INVALID_ARG;
  }
  GateBwdArgs a;
  a.u = u;
  a.v = v;
  a.G = grad_f;
  a.du = grad_u;
  a.dv = grad_v;
  a.h = plan->d_gh;
  a.psum = reinterpret_cast<float*>(plan->d_gpart);  // free once the softmax statistics are formed
  a.S = plan->d_gS;
  a.part = plan->d_gpart;
  a.fin = plan->d_gfin;
  a.scales = plan->d_bscale;
  a.B = (int)plan->B;
  a.N = (int)plan->Nu;
  a.C = (int)plan->C;
  a.events = nullptr;
  if (plan->timing_calls < plan->timing_max && (plan->timing_kind < 0 || plan->timing_kind == kKindGateBwd)) {
    plan->timing_kind = kKindGateBwd;
    a.events = &plan->events[(size_t)plan->timing_calls * kMaxEvents];
    ++plan->timing_calls;
  }
  const hipError_t e = launch_gate_bwd(plan->L, a, stream);
  if (e != hipSuccess) {
    set_error("kernel launch failed: %s", hipGetErrorString(e));
    return CGCONV_ERR_HIP;
  }
  return CGCONV_OK;
}

int64_t cgconv_paths(int32_t L_max, int32_t* l1l2J, int64_t cap) {
  if (L_max < 0 || L_max > CGCONV_LMAX) {
    set_error("unsupported L_max=%d", L_max);
    return CGCONV_ERR_UNSUPPORTED;
  }
  if (cap < 0 || (cap > 0 && !l1l2J)) {
    set_error("invalid output buffer");
    return CGCONV_ERR_INVALID_ARG;
  }
  int64_t n = 0;
  for (int l1 = 0; l1 <= L_max; ++l1)
    for (int l2 = 0; l2 <= L_max; ++l2)
      for (int J = std::abs(l1 - l2); J <= std::min(l1 + l2, (int)L_max); ++J) {
        if (n < cap) {
          l1l2J[3 * n] = l1;
          l1l2J[3 * n + 1] = l2;
          l1l2J[3 * n + 2] = J;
        }
        ++n;
      }
  return n;
}

int64_t cgconv_cg_table(int32_t L_max, int32_t* idx, double* coef, int64_t cap) {
  if (L_max < 0 || L_max > CGCONV_LMAX) {
    set_error("unsupported L_max=%d", L_max);
    return CGCONV_ERR_UNSUPPORTED;
  }
  if (cap < 0 || (cap > 0 && (!idx || !coef))) {
    set_error("invalid output buffers");
    return CGCONV_ERR_INVALID_ARG;
  }
  const std::vector<RealEntry> t = real_table(L_max);
  for (int64_t e = 0; e < (int64_t)t.size() && e < cap; ++e) {
    const RealEntry& r = t[e];
    const int32_t v[6] = {r.l1, r.m1, r.l2, r.m2, r.J, r.M};
    std::memcpy(idx + 6 * e, v, sizeof v);
    coef[e] = r.coef;
  }
  return (int64_t)t.size();
}

int cgconv_contract_host(int32_t L_max, const double* qhat, const double* khat, double* uhat) {
  if (L_max < 0 || L_max > CGCONV_LMAX) {
    set_error("unsupported L_max=%d", L_max);
    return CGCONV_ERR_UNSUPPORTED;
  }
  if (!qhat || !khat || !uhat) {
    set_error("NULL buffer");
    return CGCONV_ERR_INVALID_ARG;
  }
  contract_host(L_max, reinterpret_cast<const std::complex<double>*>(qhat),
                reinterpret_cast<const std::complex<double>*>(khat), reinterpret_cast<std::complex<double>*>(uhat));
  return CGCONV_OK;
}

}  // extern "C"

// ---- gating without allocation ---------------------------------------------
//
// cgconv_gate_value_noalloc keeps the gating partials and statistics in a
// file-scope device array instead of a plan workspace.  In host code the
// array's name is not a device address: its address on each device comes
// from hipGetSymbolAddress, taken once per device at the entry point's first
// call there, and only that address is passed to kernels.

namespace {

constexpr size_t kNoAllocScratchBytes = size_t(16) << 20;
__device__ __align__(256) float2 scratch[kNoAllocScratchBytes / sizeof(float2)];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
float2* g_scratch_ptr[kMaxDevices] = {};

// this device's copy of the array, or nullptr with the error set
float2* device_scratch(int dev) {
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      set_error("hipGetSymbolAddress of the gating scratch array failed on device %d: %s", dev,
                hipGetErrorString(e));
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[dev] = static_cast<float2*>(ptr);
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

int cgconv_gate_value_noalloc(int64_t batch, int64_t N, int32_t L_max, int64_t C, const float* u, const float* v,
                              float* f, hipStream_t stream) {
  g_last_error.clear();
  if (batch < 1 || batch > 65535 || N < 1 || C < 1 || L_max < 0) {
    set_error("invalid sizes: batch=%lld N=%lld L_max=%d C=%lld (need 1 <= batch <= 65535, N >= 1, L_max >= 0, "
              "C >= 1)", (long long)batch, (long long)N, L_max, (long long)C);
    return CGCONV_ERR_INVALID_ARG;
  }
  if (L_max > CGCONV_LMAX) {
    set_error("unsupported L_max=%d: at most %d", L_max, CGCONV_LMAX);
    return CGCONV_ERR_UNSUPPORTED;
  }
  if (!u || !v || !f) {
    set_error("u, v and f must be non-NULL device pointers");
    return CGCONV_ERR_INVALID_ARG;
  }
  if (!aligned16(u) || !aligned16(v) || !aligned16(f)) {
    set_error("u, v and f must be 16-byte aligned");
    return CGCONV_ERR_ALIGNMENT;
  }
  if (f == u || f == v) {
    set_error("f must not alias u or v");
    return CGCONV_ERR_INVALID_ARG;
  }
  const int K = (L_max + 1) * (L_max + 1);
  if ((long double)batch * N * K * C > 4.0e9L || N > INT32_MAX || C > INT32_MAX) {
    set_error("problem too large: batch*N*K*C=%.3Le (max 4e9)", (long double)batch * N * K * C);
    return CGCONV_ERR_UNSUPPORTED;
  }
  // partials [B][chunks][L+1][C] followed by the statistics [B][L+1][C]
  const long double chunks = (long double)((N + kGateChunk - 1) / kGateChunk);
  const long double need = (long double)batch * (L_max + 1) * C * (chunks + 1) * sizeof(float2);
  if (need > (long double)kNoAllocScratchBytes) {
    set_error("gating scratch of %.0Lf bytes exceeds the %zu-byte array (batch*(N/64+2)*(L_max+1)*C*8 must fit)",
              need, kNoAllocScratchBytes);
    return CGCONV_ERR_UNSUPPORTED;
  }
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    set_error("no usable current device (%d): %s", dev, hipGetErrorString(e));
    return CGCONV_ERR_HIP;
  }
  float2* base = device_scratch(dev);
  if (!base) return CGCONV_ERR_HIP;
  GateArgs a;
  a.u = u;
  a.v = v;
  a.f = f;
  a.part = base;
  a.fin = base + (size_t)batch * (size_t)chunks * (L_max + 1) * C;
  a.B = (int)batch;
  a.N = (int)N;
  a.C = (int)C;
  a.events = nullptr;
  e = launch_gate(L_max, a, stream);
  if (e != hipSuccess) {
    set_error("kernel launch failed: %s", hipGetErrorString(e));
    return CGCONV_ERR_HIP;
  }
  return CGCONV_OK;
}

}  // extern "C"
