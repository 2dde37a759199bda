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
// One thread per channel, a workgroup per (utterance, 256 channels, 8 frames): the
// thread computes the GLU of its channel over the 16 frames the window needs, in
// registers, then slides the 9 taps over them.  The GLU of every int8 pair (a, b) and
// the Swish of every int16 value with its requantization sit in tables computed once
// per handle with the formulas above (`glu_table`, 64 KB; `swish16_table`, 64 KB), so
// a GLU costs one byte load and an output its nine multiply-adds, one requantization
// and one byte load: evaluated in place, the GLU's two 64-bit products were most of
// the kernel's instructions.  8 frames per workgroup (twice the GLU work of the
// window's halo) ran the module 8 % faster than 16, and 4 or 32 frames slower; four
// channels per lane (dword loads and stores) ran it 13 % slower (a quarter of the
// waves, each holding four times the registers).  Loads and stores of a frame are 256
// consecutive elements across the workgroup.  Per frame and channel the kernel reads 2
// bytes of PW1's output (each twice, with the halo) and writes the int8 Swish output;
// the int16 BatchNorm output is written only when the launch asks for it (v != NULL:
// an inspection of the intermediate, which reruns the kernel on the kept PW1 output),
// not on a module run.
#include "ipk_internal.h"

namespace ipk {

constexpr int CONV_TAPS = 9, CONV_HALF = 4;
constexpr int CONV_FRAMES = 8;    // output frames per workgroup (the window: 16 frames in registers)
constexpr int CONV_CH = 256;      // channels per workgroup (one per thread)
constexpr int CONV_WIN = CONV_FRAMES + 2 * CONV_HALF;

struct ConvArgs {
  const int8_t* u;  // [B][T][2 d] PW1 output: a = channels [0, d), b = [d, 2 d)
  int8_t* o;        // [B][T][d]
  int16_t* v;       // [B][T][d], or NULL: not stored
  const int8_t* w;  // [d][9]
  const int32_t* bias;
  const int32_t* mult;
  const int8_t* swtab16;  // [65535]: Swish output of each int16 v, at v + 32767
  const int8_t* glutab;   // [256][256]: GLU output of (a, b), at (a + 128) 256 + b + 128
  Lengths lens;           // valid frames per utterance
  int T, d, shift_dw;
  long long glu_qc, glu_q1, m_glu;
  int shift_glu;
};

__device__ __forceinline__ long long rs64(long long a, long long m, int n) {
  return (a * m + (1ll << (n - 1))) >> n;
}

__device__ __forceinline__ long long poly_l(long long aq, long long q_c, long long q_1) {
  const long long t = (aq < q_c ? aq : q_c) - q_c;
  return t * t + q_1;
}

// The Swish of Eq. 12 on every int16 input and its requantization to PW2's int8 grid,
// one thread per value (computed once per handle; the middle kernel looks it up).
__global__ __launch_bounds__(256) void swish16_table(int8_t* tab, long long q_c, long long q_1, long long m,
                                                     int shift) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= 65535) return;
  const long long v = (long long)i - 32767;
  const long long av = v < 0 ? -v : v;
  const long long q = -(av * poly_l(av, q_c, q_1) + v * q_1);
  const long long o = rs64(q, m, shift);
  tab[i] = (int8_t)(o < -127 ? -127 : (o > 127 ? 127 : o));
}

// The GLU of every int8 pair: g = clamp8(RS(a sigma(b), m_glu, n_glu)), one thread per
// (a, b), at (a + 128) 256 + b + 128 (computed once per handle; the middle kernel looks
// it up).
__global__ __launch_bounds__(256) void glu_table(int8_t* tab, long long q_c, long long q_1, long long m, int shift) {
  const long long av = (long long)blockIdx.x - 128, bv = (long long)threadIdx.x - 128;
  const long long ab = bv < 0 ? -bv : bv;
  const long long sg = bv > 0 ? 1 : (bv < 0 ? -1 : 0);
  const long long sig = -(q_1 + sg * poly_l(ab, q_c, q_1));
  const long long r = rs64(av * sig, m, shift);
  tab[blockIdx.x * 256 + threadIdx.x] = (int8_t)(r < -127 ? -127 : (r > 127 ? 127 : r));
}

__global__ __launch_bounds__(CONV_CH) void conv_glu_dw_swish(ConvArgs a) {
  const int tid = threadIdx.x;
  const int c = blockIdx.y * CONV_CH + tid;
  const int b = blockIdx.z;
  const int t0 = blockIdx.x * CONV_FRAMES;
  const int T = a.T, d = a.d;
  if (c >= d) return;
  const int L = a.lens.len[b];
  const int8_t* ub = a.u + (size_t)b * T * 2 * d + c;
  // GLU over the window t0 - 4 .. t0 + 11, in registers (static indices)
  int g[CONV_WIN];
#pragma unroll
  for (int f = 0; f < CONV_WIN; ++f) {
    const int t = t0 - CONV_HALF + f;
    int gv = 0;
    if (t >= 0 && t < L) {
      const int av = ub[(size_t)t * 2 * d], bi = ub[(size_t)t * 2 * d + d];
      gv = a.glutab[(av + 128) * 256 + bi + 128];
    }
    g[f] = gv;
  }
  int w[CONV_TAPS];
#pragma unroll
  for (int k = 0; k < CONV_TAPS; ++k) w[k] = a.w[c * CONV_TAPS + k];
  const int bias = a.bias[c];
  const long long mdw = a.mult[c];
#pragma unroll
  for (int f = 0; f < CONV_FRAMES; ++f) {
    const int t = t0 + f;
    if (t >= T) break;
    int acc = bias;
#pragma unroll
    for (int k = 0; k < CONV_TAPS; ++k) acc += w[k] * g[f + k];
    long long vv = rs64(acc, mdw, a.shift_dw);
    vv = vv < -32767 ? -32767 : (vv > 32767 ? 32767 : vv);
    const size_t idx = ((size_t)b * T + t) * d + c;
    if (a.v) a.v[idx] = (int16_t)vv;
    a.o[idx] = t < L ? a.swtab16[vv + 32767] : (int8_t)0;
  }
}

hipError_t launch_swish16_table(int8_t* tab, long long q_c, long long q_1, long long m, int shift, hipStream_t st) {
  hipLaunchKernelGGL(swish16_table, dim3((65535 + 255) / 256), dim3(256), 0, st, tab, q_c, q_1, m, shift);
  return hipGetLastError();
}

hipError_t launch_glu_table(int8_t* tab, long long q_c, long long q_1, long long m, int shift, hipStream_t st) {
  hipLaunchKernelGGL(glu_table, dim3(256), dim3(256), 0, st, tab, q_c, q_1, m, shift);
  return hipGetLastError();
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
  a.swtab16 = m.swtab16;
  a.glutab = m.glutab;
  const dim3 grid((unsigned)((T + CONV_FRAMES - 1) / CONV_FRAMES), (unsigned)((d + CONV_CH - 1) / CONV_CH),
                  (unsigned)B);
  hipLaunchKernelGGL(conv_glu_dw_swish, grid, dim3(CONV_CH), 0, st, a);
  return hipGetLastError();
}

}  // namespace ipk
