// The element-wise and depthwise middle of the convolution module (Eq. 5):
// GLU -> depthwise convolution over time (K = 9, BatchNorm folded) -> INT16
// BatchNorm output -> Swish -> int8 input of PW2, in one pass over PW1's output.
//
// For utterance b, channel c and frame t (L = L_b, zero outside [0, L)):
//   g[t]  = clamp8(RS(a[t] sigma(b[t]), m_glu, n_glu))      a, b: the two halves of PW1's output
//   sigma = -(q_1 + sgn(b) L(b)),  L(q) = (min(|q|, q_c) - q_c)^2 + q_1   (Eq. 12's polynomial at x/2)
//   v[t]  = clamp16(RS(bias + sum_k w[k] g[t + k - 4], m_dw, n_dw))       the INT16 BatchNorm output
//   o[t]  = clamp8(RS(swish(v[t]), m_sw, n_sw)) for t < L, else 0        Eq. 12's Swish on v's grid
// Every product fits 64 bits: the host proves |a sigma| m_glu and |swish(v)| m_sw below
// 2^62 for every int8 pair and every int16 v before it accepts the constants.
//
// One thread per channel, a workgroup per (utterance, 256 channels, 64 frames): the
// thread computes the GLU of its channel over the 72 frames the window needs into its
// own LDS column (no other thread reads it, so no barrier), then slides the 9 taps.
// Loads and stores of a frame are 256 consecutive bytes across the workgroup.  The
// work is a few hundred bytes per frame and channel of integer arithmetic: the kernel
// is bound by its VALU work and the HBM traffic of PW1's output (2 d bytes per frame
// in, d + 2 d bytes out with the int16 BatchNorm output).
#include "ipk_internal.h"

namespace ipk {

constexpr int CONV_TAPS = 9, CONV_HALF = 4;
constexpr int CONV_FRAMES = 64;   // output frames per workgroup
constexpr int CONV_CH = 256;      // channels per workgroup (one per thread)

struct ConvArgs {
  const int8_t* u;  // [B][T][2 d] PW1 output: a = channels [0, d), b = [d, 2 d)
  int8_t* o;        // [B][T][d]
  int16_t* v;       // [B][T][d]
  const int8_t* w;  // [d][9]
  const int32_t* bias;
  const int32_t* mult;
  Lengths lens;  // valid frames per utterance
  int T, d, shift_dw;
  long long glu_qc, glu_q1, m_glu;
  int shift_glu;
  long long sw_qc, sw_q1, m_sw;
  int shift_sw;
};

__device__ __forceinline__ long long rs64(long long a, long long m, int n) {
  return (a * m + (1ll << (n - 1))) >> n;
}

__device__ __forceinline__ long long poly_l(long long aq, long long q_c, long long q_1) {
  const long long t = (aq < q_c ? aq : q_c) - q_c;
  return t * t + q_1;
}

__global__ __launch_bounds__(CONV_CH) void conv_glu_dw_swish(ConvArgs a) {
  __shared__ int8_t gcol[CONV_FRAMES + 2 * CONV_HALF][CONV_CH];
  const int tid = threadIdx.x;
  const int c = blockIdx.y * CONV_CH + tid;
  const int b = blockIdx.z;
  const int t0 = blockIdx.x * CONV_FRAMES;
  const int T = a.T, d = a.d;
  if (c >= d) return;
  const int L = a.lens.len[b];
  const int8_t* ub = a.u + (size_t)b * T * 2 * d;
  // GLU over the window of frames t0 - 4 .. t0 + 64 + 3
  for (int f = 0; f < CONV_FRAMES + 2 * CONV_HALF; ++f) {
    const int t = t0 - CONV_HALF + f;
    long long gv = 0;
    if (t >= 0 && t < L) {
      const long long av = ub[(size_t)t * 2 * d + c], bv = ub[(size_t)t * 2 * d + d + c];
      const long long ab = bv < 0 ? -bv : bv;
      const long long sg = bv > 0 ? 1 : (bv < 0 ? -1 : 0);
      const long long sig = -(a.glu_q1 + sg * poly_l(ab, a.glu_qc, a.glu_q1));
      gv = rs64(av * sig, a.m_glu, a.shift_glu);
      gv = gv < -127 ? -127 : (gv > 127 ? 127 : gv);
    }
    gcol[f][tid] = (int8_t)gv;
  }
  int w[CONV_TAPS];
#pragma unroll
  for (int k = 0; k < CONV_TAPS; ++k) w[k] = a.w[c * CONV_TAPS + k];
  const int bias = a.bias[c];
  const long long mdw = a.mult[c];
  const int tend = min(t0 + CONV_FRAMES, T);
  for (int t = t0; t < tend; ++t) {
    const int f = t - t0;
    int acc = bias;
#pragma unroll
    for (int k = 0; k < CONV_TAPS; ++k) acc += w[k] * (int)gcol[f + k][tid];
    long long vv = rs64(acc, mdw, a.shift_dw);
    vv = vv < -32767 ? -32767 : (vv > 32767 ? 32767 : vv);
    const size_t idx = ((size_t)b * T + t) * d + c;
    a.v[idx] = (int16_t)vv;
    long long ov = 0;
    if (t < L) {
      const long long av = vv < 0 ? -vv : vv;
      const long long q = -(av * poly_l(av, a.sw_qc, a.sw_q1) + vv * a.sw_q1);
      ov = rs64(q, a.m_sw, a.shift_sw);
      ov = ov < -127 ? -127 : (ov > 127 ? 127 : ov);
    }
    a.o[idx] = (int8_t)ov;
  }
}

hipError_t launch_conv_middle(const ConvMiddle& m, const int8_t* u, const Lengths& lens, int B, int T, int d,
                              int8_t* o, int16_t* v, hipStream_t st) {
  ConvArgs a{};
  a.u = u;
  a.o = o;
  a.v = v;
  a.w = m.w_dw;
  a.bias = m.bias_dw;
  a.mult = m.mult_dw;
  a.lens = lens;
  a.T = T;
  a.d = d;
  a.shift_dw = m.shift_dw;
  a.glu_qc = m.glu_qc;
  a.glu_q1 = m.glu_q1;
  a.m_glu = m.m_glu;
  a.shift_glu = m.shift_glu;
  a.sw_qc = m.sw_qc;
  a.sw_q1 = m.sw_q1;
  a.m_sw = m.m_sw;
  a.shift_sw = m.shift_sw;
  const dim3 grid((unsigned)((T + CONV_FRAMES - 1) / CONV_FRAMES), (unsigned)((d + CONV_CH - 1) / CONV_CH),
                  (unsigned)B);
  hipLaunchKernelGGL(conv_glu_dw_swish, grid, dim3(CONV_CH), 0, st, a);
  return hipGetLastError();
}

}  // namespace ipk
