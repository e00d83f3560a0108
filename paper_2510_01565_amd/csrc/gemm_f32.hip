// fp32 GEMM on the vector ALUs, Y = A W^T + b with the same epilogues as the
// bf16 kernel.  Used by fp32 models (no reduced-precision arithmetic at all);
// 64x64 output tiles, 256 threads with a 4x4 register block each, operands
// staged through LDS transposed to K-major so the inner loop reads float4s.
#include "device_common.h"

namespace dit {

namespace {

constexpr int TM = 64, TN = 64, TK = 64;
constexpr int LPT = TM * TK / 256;  // operand values per thread per K tile

__global__ __launch_bounds__(256) void gemm_f32_kernel(const GemmProblem P) {
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];

  const int tiles_n = (P.N + TN - 1) / TN;
  const int tm0 = (P.g[0].M + TM - 1) / TM;
  int id = blockIdx.x;
  int gi = 0;
  if (id >= tm0 * tiles_n) {
    gi = 1;
    id -= tm0 * tiles_n;
  }
  const float* __restrict__ A = (const float*)(gi ? P.g[1].A : P.g[0].A);
  const float* __restrict__ W = (const float*)(gi ? P.g[1].W : P.g[0].W);
  const long lda = gi ? P.g[1].lda : P.g[0].lda;
  const long ldw = gi ? P.g[1].ldw : P.g[0].ldw;
  const int M = gi ? P.g[1].M : P.g[0].M;
  const int K = gi ? P.g[1].K : P.g[0].K;
  const int N = P.N;
  const int m0 = (id / tiles_n) * TM, n0 = (id % tiles_n) * TN;

  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;  // 16 x 16 threads, each 4 x 4 outputs
  float acc[4][4] = {};

  // 64 rows x 64 k per operand = 4096 values, 16 per thread (64 consecutive k
  // of a row per wave).  The next K tile is loaded into registers while this
  // one is multiplied; addresses are clamped into the operands (no load behind
  // a branch, so all of them are in flight at once) and values outside them
  // replaced by zero.
  static_assert(TM == TN && TK == 64, "load mapping");
  float ra[LPT], rb[LPT];
  auto gload = [&](int k0) {
#pragma unroll
    for (int c = 0; c < LPT; ++c) {
      const int idx = tid + c * 256;
      const int row = idx >> 6, kk = idx & 63;
      const int gk = k0 + kk;
      const int am = m0 + row, bn = n0 + row;
      const float va = A[(long)min(am, M - 1) * lda + min(gk, K - 1)];
      const float vb = W[(long)min(bn, N - 1) * ldw + min(gk, K - 1)];
      ra[c] = (am < M && gk < K) ? va : 0.f;
      rb[c] = (bn < N && gk < K) ? vb : 0.f;
    }
  };
  gload(0);
  for (int k0 = 0; k0 < K; k0 += TK) {
#pragma unroll
    for (int c = 0; c < LPT; ++c) {
      const int idx = tid + c * 256;
      const int row = idx >> 6, kk = idx & 63;
      As[kk][row] = ra[c];
      Bs[kk][row] = rb[c];
    }
    __syncthreads();
    if (k0 + TK < K) gload(k0 + TK);
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      const float4 a = *(const float4*)&As[kk][ty * 4];
      const float4 b = *(const float4*)&Bs[kk][tx * 4];
      const float av[4] = {a.x, a.y, a.z, a.w};
      const float bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }

  const EpiArgs E = gi ? P.g[1].epi : P.g[0].epi;
  const float* bias = (const float*)E.bias;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
    RowEntry re;
    if (E.mode == EPI_RESID || E.mode == EPI_QKV) re = make_row_entry(P.meta, E.row_base + m);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= N) continue;
      const int jp = j ^ 1;  // partner column n ^ 1 lives in the same thread (n0 and tx*4 are even)
      const int np = n0 + tx * 4 + jp;
      const float y = acc[i][j] + (bias ? bias[n] : 0.f);
      const float yp = acc[i][jp] + ((bias && np < N) ? bias[np] : 0.f);
      epilogue_element<float>(E, re, m, n, y, yp);
    }
  }
}

}  // namespace

hipError_t launch_gemm_f32(const GemmProblem& p, hipStream_t s) {
  const int tiles_n = (p.N + TN - 1) / TN;
  long tiles = (long)((p.g[0].M + TM - 1) / TM) * tiles_n;
  if (p.n_groups > 1) tiles += (long)((p.g[1].M + TM - 1) / TM) * tiles_n;
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL(gemm_f32_kernel, dim3((unsigned)tiles), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace dit
