// bf16 GEMM on the gfx950 matrix cores: Y = A W^T + b, fp32 accumulation,
// with the step's fused epilogues (QKV scatter + 2-D RoPE, GELU, gated
// residual, plain stores).  Both operands are K-contiguous ([M, K] and
// [N, K]), which is the layout v_mfma_f32_32x32x16_bf16 wants for its A and
// B lanes (8 consecutive K values per lane), so tiles go global -> registers
// -> LDS (16-byte chunks, XOR-swizzled per row against bank conflicts) ->
// registers -> MFMA.  One launch may hold two problems ("groups") that share
// N, e.g. the text and image streams of a double-stream block, so the small
// text-stream GEMM fills otherwise idle compute units.
#include "device_common.h"

namespace dit {

namespace {

constexpr int BK = 64;  // K per stage: 8 chunks of 8 bf16 per row

struct TileCoord {
  int group, m0, n0;
};

template <int BM, int BN>
__device__ __forceinline__ TileCoord tile_coord(const GemmProblem& P) {
  const int tiles_n = (P.N + BN - 1) / BN;
  const int tm0 = (P.g[0].M + BM - 1) / BM;
  const int tiles0 = tm0 * tiles_n;
  int id = xcd_remap(blockIdx.x, gridDim.x);
  int g = 0, tm = tm0;
  if (id >= tiles0) {
    g = 1;
    id -= tiles0;
    tm = (P.g[1].M + BM - 1) / BM;
  }
  // grouped order: 8 M-tiles share each run of N-tiles, for L2 reuse of both operands
  constexpr int GM = 8;
  const int per_group = GM * tiles_n;
  const int grp = id / per_group;
  const int first_m = grp * GM;
  const int gsize = min(tm - first_m, GM);
  const int in_grp = id - grp * per_group;
  TileCoord c;
  c.group = g;
  c.m0 = (first_m + in_grp % gsize) * BM;
  c.n0 = (in_grp / gsize) * BN;
  return c;
}

template <int BM, int BN, int NWM, int NWN>
__global__ __launch_bounds__(NWM* NWN * 64) void gemm_bf16_kernel(const GemmProblem P) {
  constexpr int NT = NWM * NWN * 64;
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int A_CH = BM * 8 / NT, B_CH = BN * 8 / NT;
  static_assert(FM >= 1 && FN >= 1 && A_CH >= 1 && B_CH >= 1, "tile config");
  static_assert((BM * 8) % NT == 0 && (BN * 8) % NT == 0, "tile config");

  __shared__ uint4 lds[2][(BM + BN) * 8];

  const TileCoord tc = tile_coord<BM, BN>(P);
  const int gi = tc.group;
  const bf16_t* __restrict__ A = (const bf16_t*)(gi ? P.g[1].A : P.g[0].A);
  const bf16_t* __restrict__ W = (const bf16_t*)(gi ? P.g[1].W : P.g[0].W);
  const long lda = gi ? P.g[1].lda : P.g[0].lda;
  const long ldw = gi ? P.g[1].ldw : P.g[0].ldw;
  const int M = gi ? P.g[1].M : P.g[0].M;
  const int K = gi ? P.g[1].K : P.g[0].K;
  const int N = P.N;
  const int m0 = tc.m0, n0 = tc.n0;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / NWN, wn = wave % NWN;

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  uint4 ra[A_CH], rb[B_CH];
  const int KT = (K + BK - 1) / BK;

  // Global loads: addresses are clamped into the operand so every load is
  // issued unconditionally; out-of-range chunks are replaced by zeros.
  auto gload = [&](int kt) {
    const int k0 = kt * BK;
#pragma unroll
    for (int c = 0; c < A_CH; ++c) {
      const int idx = tid + c * NT;
      const int row = idx >> 3, kc = idx & 7;
      const int gr = m0 + row, gk = k0 + kc * 8;
      const bool ok = gr < M && gk < K;
      const uint4 v = *(const uint4*)(A + (long)min(gr, M - 1) * lda + min(gk, K - 8));
      ra[c] = ok ? v : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < B_CH; ++c) {
      const int idx = tid + c * NT;
      const int row = idx >> 3, kc = idx & 7;
      const int gr = n0 + row, gk = k0 + kc * 8;
      const bool ok = gr < N && gk < K;
      const uint4 v = *(const uint4*)(W + (long)min(gr, N - 1) * ldw + min(gk, K - 8));
      rb[c] = ok ? v : make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int st) {
#pragma unroll
    for (int c = 0; c < A_CH; ++c) {
      const int idx = tid + c * NT;
      const int row = idx >> 3, kc = idx & 7;
      lds[st][row * 8 + (kc ^ (row & 7))] = ra[c];
    }
#pragma unroll
    for (int c = 0; c < B_CH; ++c) {
      const int idx = tid + c * NT;
      const int row = idx >> 3, kc = idx & 7;
      lds[st][(BM + row) * 8 + (kc ^ (row & 7))] = rb[c];
    }
  };
  // fragments of k-step ks (16 wide) of stage st: lane row (lane & 31), chunk 2 ks + lane / 32
  bf16x8_t fa[2][FM], fb[2][FN];
  auto fload = [&](int st, int ks, int buf) {
    const int ch = ks * 2 + (lane >> 5);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WTM + i * 32 + (lane & 31);
      fa[buf][i] = __builtin_bit_cast(bf16x8_t, lds[st][row * 8 + (ch ^ (row & 7))]);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int row = wn * WTN + j * 32 + (lane & 31);
      fb[buf][j] = __builtin_bit_cast(bf16x8_t, lds[st][(BM + row) * 8 + (ch ^ (row & 7))]);
    }
  };

  gload(0);
  lstore(0);
  __syncthreads();

  for (int kt = 0; kt < KT; ++kt) {
    const int st = kt & 1;
    if (kt + 1 < KT) gload(kt + 1);
    fload(st, 0, 0);
    static_for<BK / 16>([&](auto kk) {
      constexpr int ks = decltype(kk)::value;
      constexpr int cur = ks & 1;
      if constexpr (ks + 1 < BK / 16) fload(st, ks + 1, cur ^ 1);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][i], fb[cur][j], acc[i][j], 0, 0, 0);
    });
    if (kt + 1 < KT) lstore(st ^ 1);
    __syncthreads();
  }

  // epilogue.  Row facts (request, joint position, grid position) are computed
  // once per tile row into LDS, so the unrolled element loop never indexes the
  // batch metadata.
  RowEntry* rows = (RowEntry*)&lds[0][0];
  static_assert(BM * sizeof(RowEntry) <= sizeof(lds), "row table");
  const EpiArgs E = gi ? P.g[1].epi : P.g[0].epi;
  if (E.mode == EPI_RESID || E.mode == EPI_QKV) {
    for (int t = tid; t < BM; t += NT)
      if (m0 + t < M) rows[t] = make_row_entry(P.meta, E.row_base + m0 + t);
    __syncthreads();
  }
  const bf16_t* bias = (const bf16_t*)E.bias;
  static_for<FN>([&](auto jj) {
    constexpr int j = decltype(jj)::value;
    const int n = n0 + wn * WTN + j * 32 + (lane & 31);
    const float bn = (bias != nullptr && n < N) ? bf2f(bias[n]) : 0.f;
    static_for<FM>([&](auto ii) {
      constexpr int i = decltype(ii)::value;
      static_for<16>([&](auto rr) {
        constexpr int r = decltype(rr)::value;
        const int ml = wm * WTM + i * 32 + (r / 4) * 8 + (lane >> 5) * 4 + (r % 4);
        const int m = m0 + ml;
        const float y = acc[i][j][r] + bn;
        const float yp = __shfl_xor(y, 1, 64);
        if (m < M && n < N) {
          RowEntry re;
          if (E.mode == EPI_RESID || E.mode == EPI_QKV) re = rows[ml];
          epilogue_element<bf16_t>(E, re, m, n, y, yp);
        }
      });
    });
  });
}

template <int BM, int BN, int NWM, int NWN>
hipError_t launch_cfg(const GemmProblem& p, hipStream_t s) {
  const int tiles_n = (p.N + BN - 1) / BN;
  long tiles = (long)((p.g[0].M + BM - 1) / BM) * tiles_n;
  if (p.n_groups > 1) tiles += (long)((p.g[1].M + BM - 1) / BM) * tiles_n;
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, NWM, NWN>), dim3((unsigned)tiles), dim3(NWM * NWN * 64), 0, s,
                     p);
  return hipGetLastError();
}

}  // namespace

namespace {
enum GemmCfg { CFG_128x64 = 0, CFG_256x128 = 1, CFG_128x128 = 2 };
GemmCfg pick(const GemmProblem& p) {
  int maxM = p.g[0].M;
  if (p.n_groups > 1 && p.g[1].M > maxM) maxM = p.g[1].M;
  if (p.N <= 64) return CFG_128x64;
  if (maxM >= 2048 && p.N >= 1024) return CFG_256x128;
  return CFG_128x128;
}
}  // namespace

const char* gemm_bf16_config_name(const GemmProblem& p) {
  static const char* names[] = {"gemm_bf16_128x64", "gemm_bf16_256x128", "gemm_bf16_128x128"};
  return names[pick(p)];
}

hipError_t launch_gemm_bf16(const GemmProblem& p, hipStream_t s) {
  switch (pick(p)) {
    case CFG_128x64:
      return launch_cfg<128, 64, 4, 1>(p, s);
    case CFG_256x128:
      return launch_cfg<256, 128, 2, 2>(p, s);
    default:
      return launch_cfg<128, 128, 2, 2>(p, s);
  }
}

}  // namespace dit
