// Inter-channel CG stage with a per-degree channel reduction, for gfx950
// (arXiv 2509.24093 §4.1: within a head every query channel c1 meets every
// key channel c2, (2J+1) m m components per degree, and the multiplicity is
// reduced by a learned equivariant map, read as one matrix per head and
// output degree):
//
//   out[(J,M), h m_o + o] = sum_{c1,c2} W[h][J][o][c1 m + c2] u[(J,M), h, c1, c2]
//
// at every frequency, u being the CG product of the spectra of query channel
// h m + c1 and key channel h m + c2 (the reduction is linear, so it commutes
// with the inverse transform).  Runs between the unfused forward passes and
// the unfused inverse passes.
//
// Block = one batch element, one head and 4 frequency points w in [0, N/2];
// lane = (point, pair slot c1*8 + c2), 64 slots per point (m <= 8; a slot
// with c1 or c2 >= m meets zero weights).  The block loads the head's
// spectra at w and N - w of its points into LDS once.  Each lane forms 2Q of
// channel h m + c1 in registers; 2K of every key channel is formed once per
// point, in the complex-m basis, and stays in LDS, where the eight lanes of a
// key channel read it (broadcast) block by block of the generated
// contraction (CgBody with an LDS key operand).  With the key operand out of
// the registers a lane needs 166 VGPRs instead of 256, so three waves share
// a SIMD instead of two.
// Every output component is parked in LDS per output phase; after the phase
// the matrix cores reduce the 64 pair values of each component with the
// degree's matrix, v_mfma_f32_16x16x4f32 in fp32 (A: rows o padded to 16,
// columns 4 pair slots per step, 16 steps; B: the parked values, columns
// (point, sign of M, re/im)), and the packed output W = U_o + i U_{o+1}
// goes to row w, conj U_o + i conj U_{o+1} to row N - w.
#include <hip/hip_runtime.h>

#include "cg_common.h"

namespace cgconv {
namespace cgdev {
#include CGCONV_BODY
}  // namespace cgdev

namespace {

using cgdev::CgBody;
using cgdev::swap_pair;
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kPts = 4;      // frequency points per block
constexpr int kSlots = 64;   // channel-pair slots per point
constexpr int kThreadsI = kPts * kSlots;
constexpr int kWRows = kInterMmax;  // rows o of the reduction matrices held in LDS (m_out <= m)

// The key spectra of the block's points in LDS ([pt][k][c2], complex-m
// basis): the lanes of a point share them, eight lanes per key channel, and
// the eight key channels of a component are 64 contiguous bytes.
typedef float v2f __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) const v2f lds_cf2;
struct LdsKey {
  lds_cf2* p;  // this lane's key channel at component 0
  __device__ __forceinline__ float2 operator[](int k) const {
    const v2f v = p[k * kInterMmax];
    return make_float2(v.x, v.y);
  }
};
// A fresh, opaque copy per block of the contraction: the block's loads are
// not merged with another block's, so no key value stays live in a register
// beyond its block.
__device__ __forceinline__ LdsKey cg_kfence(const LdsKey& k) {
  LdsKey r = k;
  asm volatile("" : "+v"(r.p));
  return r;
}

template <int L>
struct InterGeo {
  static constexpr int K = (L + 1) * (L + 1);
  static constexpr int PMAX = L == 0 ? 1 : 2 * L;  // most components in one output phase
};

template <int L>
struct InterStore {
  static constexpr int PMAX = InterGeo<L>::PMAX;
  static constexpr int K = InterGeo<L>::K;
  float2* T;        // LDS [PMAX][kSlots][kPts]: parked outputs of the current phase
  const float* Wl;  // LDS [L+1][kWRows][kSlots]: the head's matrices (rows o >= kWRows of the MFMA operand are zero)
  char* Wb;         // packed output spectra of this batch element (bytes)
  long long N;
  int n1_log2, n2_log2, F, w0, Cpo, co0, mo;
  int slot, pt, lane, wave;

  // storage row of frequency w (rows as in the unfused CG stage)
  __device__ __forceinline__ long long row_of(long long w) const {
    return ((w & ((1LL << n1_log2) - 1)) << n2_log2) | (w >> n1_log2);
  }

  // component kout = J^2 + J + M of phase mu = |M|: slot ci within the
  // phase is J for mu = 0, 2 (J - mu) + (M < 0) otherwise
  __device__ __forceinline__ void operator()(int kout, float2 u) const {
    const int J = (int)__builtin_sqrtf((float)kout + 0.5f);
    const int M = kout - J * J - J, mu = M < 0 ? -M : M;
    const int ci = mu == 0 ? J : 2 * (J - mu) + (M < 0 ? 1 : 0);
    T[(ci * kSlots + slot) * kPts + pt] = u;
  }

  __device__ __forceinline__ void end_phase(int mu) const {
    __syncthreads();  // every lane has parked its outputs
    const int col = lane & 15, cpt = col >> 2, sgn = (col >> 1) & 1, ri = col & 1;
    const int kq = lane >> 4;  // pair slot within a step of 4; also the row group of D
    const long long w = (long long)w0 + cpt;
    const bool has = mu > 0 || sgn == 0;  // the degree-0 phase has one sign only
    for (int J = mu + wave; J <= L; J += 4) {
      const int ci = has ? (mu == 0 ? J : 2 * (J - mu) + sgn) : 0;
      v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int step = 0; step < kSlots / 4; ++step) {
        const int k = 4 * step + kq;
        const float av = col < kWRows ? Wl[(J * kWRows + col) * kSlots + k] : 0.f;  // A[o = col][pair k]
        const float2 t = T[(ci * kSlots + k) * kPts + cpt];
        const float bv = has ? (ri ? t.y : t.x) : 0.f;    // B[pair k][col]
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
      }
      // this lane holds D[o = 4 kq + i][col], i = 0..3; lane ^ 1 holds the
      // other part (re/im) of the same complex value
      float other[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) other[i] = swap_pair(acc[i]);
      const long long wn = (N - w) & (N - 1);
      const bool store = has && w < F && !(ri == 1 && wn == w);  // one row for w = 0, N/2
      if (!store) continue;
      const int kout = J * J + J + (sgn ? -mu : mu);
      const long long row = row_of(ri == 0 ? w : wn);
      float2* dst = reinterpret_cast<float2*>(Wb) + (row * K + kout) * Cpo;
#pragma unroll
      for (int i = 0; i < 4; i += 2) {
        const int o = 4 * kq + i;  // even: the channel pair (o, o + 1)
        if (o >= mo) continue;
        const float2 u0 = ri == 0 ? make_float2(acc[i], other[i]) : make_float2(other[i], acc[i]);
        const float2 u1 = ri == 0 ? make_float2(acc[i + 1], other[i + 1]) : make_float2(other[i + 1], acc[i + 1]);
        // row w: U_o + i U_{o+1};  row N - w: conj U_o + i conj U_{o+1}
        const float2 v = ri == 0 ? make_float2(u0.x - u1.y, u0.y + u1.x) : make_float2(u0.x + u1.y, u1.x - u0.y);
        dst[(co0 + o) >> 1] = v;
      }
    }
    __syncthreads();  // the next phase overwrites T
  }
};

template <int L>
__global__ __launch_bounds__(kThreadsI, 3) void cg_inter_kernel(InterArgs a) {
  constexpr int K = InterGeo<L>::K, PMAX = InterGeo<L>::PMAX;
  // the spectra of the block's points ([pt][w or N - w][k][channel of the
  // head], 2 kPts K kInterMmax values) until every lane has gathered its
  // own, then the parked outputs of the output phases
  constexpr int ZE = 2 * kPts * K * kInterMmax;
  __shared__ float2 sT[PMAX * kSlots * kPts > ZE ? PMAX * kSlots * kPts : ZE];
  __shared__ float sW[(L + 1) * kWRows * kSlots];
  __shared__ float2 sK[kPts * K * kInterMmax];
  const int tid = threadIdx.x;
  const int ngroups = (a.F + kPts - 1) / kPts;
  const int g = blockIdx.x % ngroups, bh = blockIdx.x / ngroups;
  const int h = bh % a.H, b = bh / a.H;
  const int slot = tid & (kSlots - 1), pt = tid / kSlots;
  const int c1 = slot >> 3, c2 = slot & 7;
  const long long w = (long long)g * kPts + pt;
  const bool valid = w < a.F && c1 < a.m && c2 < a.m;
  // the head's matrices, rows o < mo and slots of real pairs, zeros elsewhere
  for (int idx = tid; idx < (L + 1) * kWRows * kSlots; idx += kThreadsI) {
    const int J = idx / (kWRows * kSlots), o = (idx / kSlots) % kWRows, s = idx % kSlots;
    const int s1 = s >> 3, s2 = s & 7;
    sW[idx] = (o < a.mo && s1 < a.m && s2 < a.m)
                  ? a.wt[(((long long)h * (L + 1) + J) * a.mo + o) * a.m * a.m + s1 * a.m + s2]
                  : 0.f;
  }
  auto rowp = [&](long long x) {
    return ((x & ((1LL << a.n1_log2) - 1)) << a.n2_log2) | (x >> a.n1_log2);
  };
  // the head's spectra at w and N - w of the block's points, loaded once
  // per block (64 contiguous bytes per row and component), four loads per
  // thread in flight; points past N/2 read row 0, channels past m read zero
  {
    const float2* Zb = a.Z + (long long)b * a.N * K * a.C + (long long)h * a.m;
    constexpr int NB = 4;
    for (int base = 0; base < ZE; base += NB * kThreadsI) {
      float2 v[NB];
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const int idx = base + u * kThreadsI + tid;
        const int ch = idx % kInterMmax, k = (idx / kInterMmax) % K, side = (idx / (kInterMmax * K)) & 1,
                  pl = idx / (2 * kInterMmax * K);
        const long long wp = (long long)g * kPts + pl;
        const long long wv = wp < a.F ? wp : 0;
        const long long row = rowp(side ? (a.N - wv) & (a.N - 1) : wv);
        v[u] = (idx < ZE && ch < a.m) ? Zb[(row * K + k) * a.C + ch] : make_float2(0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const int idx = base + u * kThreadsI + tid;
        if (idx < ZE) sT[idx] = v[u];
      }
    }
  }
  __syncthreads();
  // 2K of every key channel of the block's points, in the complex-m basis,
  // into sK; each lane's 2Q into registers
  for (int idx = tid; idx < kPts * K * kInterMmax; idx += kThreadsI) {
    const int ch = idx % kInterMmax, k = (idx / kInterMmax) % K, pl = idx / (kInterMmax * K);
    const int l = (int)__builtin_sqrtf((float)k + 0.5f), m = k - l * l - l;
    auto key2 = [&](int kk) {
      const float2 A = sT[((pl * 2 + 0) * K + kk) * kInterMmax + ch], B = sT[((pl * 2 + 1) * K + kk) * kInterMmax + ch];
      return make_float2(A.y + B.y, B.x - A.x);
    };
    float2 v;
    if (m == 0) {
      v = key2(k);
    } else {
      const int mu = m < 0 ? -m : m;
      const float2 xc = key2(l * l + l + mu), xs = key2(l * l + l - mu);
      v = m < 0 ? make_float2(xc.x - xs.y, xc.y + xs.x) : make_float2(xc.x + xs.y, xc.y - xs.x);
    }
    const bool kv = (long long)g * kPts + pl < a.F && ch < a.m;
    sK[idx] = kv ? v : make_float2(0.f, 0.f);
  }
  float2 qa[K];
  {
    const float2* z1a = sT + ((pt * 2 + 0) * K) * kInterMmax + c1;
    const float2* z1b = sT + ((pt * 2 + 1) * K) * kInterMmax + c1;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const float2 A1 = z1a[k * kInterMmax], B1 = z1b[k * kInterMmax];
      qa[k] = valid ? make_float2(A1.x + B1.x, A1.y - B1.y) : make_float2(0.f, 0.f);  // 2Q of channel c1
      asm volatile("" : "+v"(qa[k].x), "+v"(qa[k].y));
    }
  }
  __syncthreads();  // every lane has gathered and sK is complete: the output phases reuse sT
  // 2Q into the complex-m basis (the basis change of the other kernels, on one operand)
#pragma unroll
  for (int l = 1; l * l < K; ++l) {
#pragma unroll
    for (int mu = 1; mu <= l; ++mu) {
      const int c = l * l + l + mu, s = l * l + l - mu;
      const float2 xc = qa[c], xs = qa[s];
      qa[s] = make_float2(xc.x - xs.y, xc.y + xs.x);
      qa[c] = make_float2(xc.x + xs.y, xc.y - xs.x);
    }
  }
  const LdsKey ka{(lds_cf2*)(sK + pt * K * kInterMmax + c2)};
  InterStore<L> st;
  st.T = sT;
  st.Wl = sW;
  st.Wb = reinterpret_cast<char*>(a.W + (long long)b * a.N * K * a.Cpo);
  st.N = a.N;
  st.n1_log2 = a.n1_log2;
  st.n2_log2 = a.n2_log2;
  st.F = a.F;
  st.w0 = g * kPts;
  st.Cpo = a.Cpo;
  st.co0 = h * a.mo;
  st.mo = a.mo;
  st.slot = slot;
  st.pt = pt;
  st.lane = tid & 63;
  st.wave = tid >> 6;
  CgBody<L>::run(qa, ka, st);
}

}  // namespace

template <>
hipError_t launch_cg_inter<CGCONV_TU_L>(const InterArgs& a, hipStream_t s) {
  if (a.m < 1 || a.m > kInterMmax || a.mo < 2 || a.mo > kWRows || (a.mo & 1) || a.C != a.H * a.m || a.F < 1)
    return hipErrorInvalidValue;
  const long long blocks = (long long)a.B * a.H * ((a.F + kPts - 1) / kPts);
  hipLaunchKernelGGL(cg_inter_kernel<CGCONV_TU_L>, dim3((unsigned)blocks), dim3(kThreadsI), 0, s, a);
  return hipGetLastError();
}

}  // namespace cgconv
