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

// LDS slot of 16-byte chunk `kc` (0..7) of tile row `row`: rows are 128 bytes,
// the XOR spreads the rows that one ds_read_b128 serves together over all banks.
template <int SWZ>
__device__ __forceinline__ int lds_slot(int row, int kc) {
  if constexpr (SWZ == 0) return row * 8 + (kc ^ (row & 7));
  else return row * 8 + (kc ^ ((row >> 1) & 7));
}

template <int BM, int BN, int NWM, int NWN, int SWZ = 1, int PF = 1, int PRIO = 0, int SGB = 0, int SB = 0>
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

  // PF register sets of the next tiles: tile t is loaded into set t % PF
  uint4 ra[PF][A_CH], rb[PF][B_CH];
  const int KT = (K + BK - 1) / BK;

  // Global loads: addresses are clamped into the operand so every load is
  // issued unconditionally; out-of-range chunks are replaced by zeros.
  auto gload = [&](int kt, auto set) {
    constexpr int S = decltype(set)::value;
    const int k0 = kt * BK;
#pragma unroll
    for (int c = 0; c < A_CH; ++c) {
      const int idx = tid + c * NT;
      const int row = idx >> 3, kc = idx & 7;
      const int gr = m0 + row, gk = k0 + kc * 8;
      const bool ok = gr < M && gk < K;
      const uint4 v = *(const uint4*)(A + (long)min(gr, M - 1) * lda + min(gk, K - 8));
      ra[S][c] = ok ? v : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < B_CH; ++c) {
      const int idx = tid + c * NT;
      const int row = idx >> 3, kc = idx & 7;
      const int gr = n0 + row, gk = k0 + kc * 8;
      const bool ok = gr < N && gk < K;
      const uint4 v = *(const uint4*)(W + (long)min(gr, N - 1) * ldw + min(gk, K - 8));
      rb[S][c] = ok ? v : make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int st, auto set) {
    constexpr int S = decltype(set)::value;
#pragma unroll
    for (int c = 0; c < A_CH; ++c) {
      const int idx = tid + c * NT;
      const int row = idx >> 3, kc = idx & 7;
      lds[st][lds_slot<SWZ>(row, kc)] = ra[S][c];
    }
#pragma unroll
    for (int c = 0; c < B_CH; ++c) {
      const int idx = tid + c * NT;
      const int row = idx >> 3, kc = idx & 7;
      lds[st][lds_slot<SWZ>(BM + row, kc)] = rb[S][c];
    }
  };
  // fragments of k-step ks (16 wide) of stage st: lane row (lane & 31), chunk 2 ks + lane / 32
  bf16x8_t fa[2][FM], fb[2][FN];
  auto fload = [&](int st, int ks, int buf) {
    const int ch = ks * 2 + (lane >> 5);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WTM + i * 32 + (lane & 31);
      fa[buf][i] = __builtin_bit_cast(bf16x8_t, lds[st][lds_slot<SWZ>(row, ch)]);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int row = wn * WTN + j * 32 + (lane & 31);
      fb[buf][j] = __builtin_bit_cast(bf16x8_t, lds[st][lds_slot<SWZ>(BM + row, ch)]);
    }
  };
  auto compute = [&](int st) {
    fload(st, 0, 0);
    static_for<BK / 16>([&](auto kk) {
      constexpr int ks = decltype(kk)::value;
      constexpr int cur = ks & 1;
      if constexpr (ks + 1 < BK / 16) fload(st, ks + 1, cur ^ 1);
      // SB: keep the next k-step's fragment reads ahead of this k-step's MFMAs
      if constexpr (SB) __builtin_amdgcn_sched_barrier(0);
      if constexpr (PRIO) __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][i], fb[cur][j], acc[i][j], 0, 0, 0);
      if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
      if constexpr (SB) __builtin_amdgcn_sched_barrier(0);
      if constexpr (SGB) {
        // one fragment read of the next k-step between consecutive MFMAs
        constexpr int NR = (ks + 1 < BK / 16) ? FM + FN : 0;
        static_for<NR>([&](auto) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        });
        __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - NR, 0);
      }
    });
  };
  // one K tile: prefetch tile kt + PF into the set that held tile kt, compute
  // tile kt from LDS, then stage tile kt + 1 into the other LDS buffer
  auto iter = [&](int kt, auto set) {
    constexpr int S = decltype(set)::value;
    if (kt + PF < KT) gload(kt + PF, set);
    compute(kt & 1);
    if (kt + 1 < KT) lstore((kt + 1) & 1, std::integral_constant<int, (S + 1) % PF>{});
    __syncthreads();
  };

  gload(0, std::integral_constant<int, 0>{});
  if constexpr (PF > 1)
    if (KT > 1) gload(1, std::integral_constant<int, 1 % PF>{});
  lstore(0, std::integral_constant<int, 0>{});
  __syncthreads();
  if constexpr (PF == 1) {
    for (int kt = 0; kt < KT; ++kt) iter(kt, std::integral_constant<int, 0>{});
  } else {
    for (int kt = 0; kt < KT; kt += 2) {
      iter(kt, std::integral_constant<int, 0>{});
      if (kt + 1 < KT) iter(kt + 1, std::integral_constant<int, 1>{});
    }
  }

  // epilogue.  Row facts (request, joint position, grid position) are computed
  // once per tile row into LDS, so the unrolled loops never index the batch
  // metadata.  Each 32x32 accumulator fragment is staged through a per-wave
  // LDS buffer so that a lane ends up with 16 consecutive columns of one row
  // and stores them with 16-byte writes.
  RowEntry* rows = (RowEntry*)&lds[0][0];
  constexpr int SP = 36;  // staging row pitch in floats (16-byte aligned rows)
  float* stg = (float*)&lds[0][0] + BM * (sizeof(RowEntry) / 4) + wave * 32 * SP;
  static_assert(BM * sizeof(RowEntry) + NWM * NWN * 32 * SP * 4 <= sizeof(lds), "epilogue LDS");
  const EpiArgs E = gi ? P.g[1].epi : P.g[0].epi;
  const bool need_rows = E.mode == EPI_RESID || E.mode == EPI_QKV;
  if (need_rows) {
    for (int t = tid; t < BM; t += NT)
      if (m0 + t < M) rows[t] = make_row_entry(P.meta, E.row_base + m0 + t);
    __syncthreads();
  }
  const bf16_t* bias = (const bf16_t*)E.bias;
  const int rl = lane >> 1, cseg = (lane & 1) * 16;
  static_for<FN>([&](auto jj) {
    constexpr int j = decltype(jj)::value;
    const int nb = n0 + wn * WTN + j * 32;
    const int nl = nb + (lane & 31);
    const float bn = (bias != nullptr && nl < N) ? bf2f(bias[nl]) : 0.f;
    static_for<FM>([&](auto ii) {
      constexpr int i = decltype(ii)::value;
      static_for<16>([&](auto rr) {
        constexpr int r = decltype(rr)::value;
        stg[((r / 4) * 8 + (lane >> 5) * 4 + (r % 4)) * SP + (lane & 31)] = acc[i][j][r] + bn;
      });
      float v[16];
      static_for<4>([&](auto qq) {
        constexpr int q = decltype(qq)::value;
        const float4 t = *(const float4*)&stg[rl * SP + cseg + 4 * q];
        v[4 * q] = t.x;
        v[4 * q + 1] = t.y;
        v[4 * q + 2] = t.z;
        v[4 * q + 3] = t.w;
      });
      const int ml = wm * WTM + i * 32 + rl;
      const int m = m0 + ml, n = nb + cseg;
      if (m < M) {
        RowEntry re;
        if (need_rows) re = rows[ml];
        if (n + 16 <= N) {
          epilogue_segment16<bf16_t>(E, re, m, n, v);
        } else {
#pragma unroll
          for (int q = 0; q < 16; ++q)
            if (n + q < N) epilogue_element<bf16_t>(E, re, m, n + q, v[q], v[q ^ 1]);
        }
      }
    });
  });
}

template <int BM, int BN, int NWM, int NWN, int SWZ = 1, int PF = 1, int PRIO = 0, int SGB = 0, int SB = 0>
hipError_t launch_cfg(const GemmProblem& p, hipStream_t s) {
  const int tiles_n = (p.N + BN - 1) / BN;
  long tiles = (long)((p.g[0].M + BM - 1) / BM) * tiles_n;
  if (p.n_groups > 1) tiles += (long)((p.g[1].M + BM - 1) / BM) * tiles_n;
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, NWM, NWN, SWZ, PF, PRIO, SGB, SB>), dim3((unsigned)tiles), dim3(NWM * NWN * 64), 0, s,
                     p);
  return hipGetLastError();
}

}  // namespace

namespace {
enum GemmCfg { CFG_128x64 = 0, CFG_256x256 = 1, CFG_128x128 = 2 };
GemmCfg pick(const GemmProblem& p) {
  int maxM = p.g[0].M;
  if (p.n_groups > 1 && p.g[1].M > maxM) maxM = p.g[1].M;
  if (p.N <= 64) return CFG_128x64;
  if (maxM >= 1024 && p.N >= 1024) return CFG_256x256;
  return CFG_128x128;
}
}  // namespace

const char* gemm_bf16_config_name(const GemmProblem& p) {
  static const char* names[] = {"gemm_bf16_128x64", "gemm_bf16_256x256", "gemm_bf16_128x128"};
  return names[pick(p)];
}

hipError_t launch_gemm_bf16(const GemmProblem& p, hipStream_t s) {
  switch (pick(p)) {
    case CFG_128x64:
      return launch_cfg<128, 64, 4, 1>(p, s);
    case CFG_256x256:
      return launch_cfg<256, 256, 2, 4>(p, s);
    default:
      return launch_cfg<128, 128, 2, 2>(p, s);
  }
}

}  // namespace dit
