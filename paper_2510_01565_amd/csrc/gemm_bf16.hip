// bf16 GEMM on the gfx950 matrix cores: Y = A W^T + b, fp32 accumulation,
// with the step's fused epilogues (QKV scatter + 2-D RoPE, GELU, gated
// residual, plain stores).
//
// Both operands are K-contiguous ([M, K] and [N, K]), which is the layout
// v_mfma_f32_32x32x16_bf16 wants for its A and B lanes (8 consecutive K values
// per lane).  Tiles move global -> LDS -> registers -> MFMA:
//  * when K is a multiple of the K tile, with direct-to-LDS loads
//    (global_load_lds_dwordx4: each wave instruction writes 64 x 16 bytes of
//    LDS without passing through registers) into a ring of STAGES buffers, so
//    the loads of tile k + STAGES - 1 are in flight while tile k is multiplied;
//  * otherwise through registers into two buffers, zero-filling the K tail.
// LDS rows are XOR-swizzled per 16-byte chunk so that the 16 rows one
// ds_read_b128 serves per cycle hit all 64 banks.  Blocks are remapped so
// every XCD owns one contiguous range of output tiles (its L2 keeps the
// operand panels those tiles share), in a grouped-M order.  One launch may
// hold two problems ("groups") sharing N -- the text and image streams of a
// double-stream block -- so the small text GEMM fills otherwise idle CUs.
#include "device_common.h"

namespace dit {

namespace {

// k-steps over which the loads of one K tile are spread (direct-to-LDS path)
constexpr int kLoadSplitK = 1;
// main-loop schedule of the direct-to-LDS path (0: one barrier per K tile, 1: whole-tile register prefetch)
constexpr int kSchedK = 1;
// chunks in which the loads of one K tile leave (whole-tile prefetch schedule)
constexpr int kLoadChunksK = 2;
// 16x16x32 MFMAs in the whole-tile prefetch schedule (else 32x32x16)
constexpr bool kMfma16K = true;

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

// LDS slot (in 16-byte chunks) of chunk `kc` of tile row `row` for rows of
// CPR chunks.  64 banks of 4 bytes serve 16 lanes of a ds_read_b128 per cycle:
// the 16 consecutive rows read at one chunk index must cover all banks.
template <int CPR>
__device__ __forceinline__ int lds_slot(int row, int kc) {
  if constexpr (CPR == 8) return row * 8 + (kc ^ ((row >> 1) & 7));  // 128-byte rows: pairs of rows share 64 banks
  else return row * 4 + (kc ^ ((row >> 2) & 3));                      // 64-byte rows: quads of rows share 64 banks
}

// s_waitcnt with vmcnt = n and the other counters left alone (gfx9 encoding:
// vmcnt[3:0] and [15:14], expcnt[6:4], lgkmcnt[11:8]).
// Word 3 of a raw buffer resource on gfx9-family targets: 32-bit data format,
// so untyped dword loads are range-checked against num_records and return
// zeros past it.
constexpr int kBufferWord3 = 0x00020000;

template <int n>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(n >= 0 && n < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <int BM, int BN, int NWM, int NWN, int BK, int STAGES, bool DTL>
__global__ __launch_bounds__(NWM* NWN * 64) void gemm_bf16_kernel(const GemmProblem P) {
  constexpr int NT = NWM * NWN * 64;
  constexpr int NWAVES = NWM * NWN;
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int CPR = BK / 8;                     // 16-byte chunks per tile row
  constexpr int STAGE = (BM + BN) * CPR;          // uint4 per stage
  static_assert(FM >= 1 && FN >= 1 && (BK == 32 || BK == 64) && STAGES >= 2 && BK % 32 == 0, "tile config");
  static_assert(STAGES * STAGE * 16 <= 160 * 1024, "LDS");

  __shared__ uint4 lds[STAGES * STAGE];

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

  // 16x16x32 MFMAs (the whole-tile-prefetch direct-to-LDS path only): the
  // 32x32 fragment (i, j) is the 2 x 2 block of 16x16 accumulators 2i.., 2j..
  constexpr bool M16 = kMfma16K && DTL && kSchedK == 1;
  f32x4_t acc16[M16 ? 2 * FM : 1][M16 ? 2 * FN : 1];
  if constexpr (M16) {
#pragma unroll
    for (int i = 0; i < 2 * FM; ++i)
#pragma unroll
      for (int j = 0; j < 2 * FN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc16[i][j][r] = 0.f;
  }
  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int KT = (K + BK - 1) / BK;

  // fragments of k-step ks (16 wide) of stage st: lane row (lane & 31), chunk 2 ks + lane / 32
  bf16x8_t fa[2][FM], fb[2][FN];
  auto fload = [&](int st, int ks, int buf) {
    const int ch = ks * 2 + (lane >> 5);
    const uint4* S = lds + st * STAGE;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WTM + i * 32 + (lane & 31);
      fa[buf][i] = __builtin_bit_cast(bf16x8_t, S[lds_slot<CPR>(row, ch)]);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int row = wn * WTN + j * 32 + (lane & 31);
      fb[buf][j] = __builtin_bit_cast(bf16x8_t, S[lds_slot<CPR>(BM + row, ch)]);
    }
  };
  auto compute = [&](int st) {
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
    // Instruction order for the scheduler: the first k-step's fragment reads,
    // then each k-step's MFMAs alternating with the next k-step's reads, so
    // LDS latency hides under the matrix cores inside every wave.
    constexpr int NR = FM + FN, NM = FM * FN, NP = NR < NM ? NR : NM;
    __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);  // DS read
    static_for<BK / 16 - 1>([&](auto) {
      static_for<NP>([&](auto) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      });
      if constexpr (NM > NP) __builtin_amdgcn_sched_group_barrier(0x008, NM - NP, 0);
      if constexpr (NR > NP) __builtin_amdgcn_sched_group_barrier(0x100, NR - NP, 0);
    });
    __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
  };

  if (DTL) {  // a compile-time constant: the other path is dropped
    // ---- direct-to-LDS ring.  LDS holds [A stage 0 .. STAGES-1 | B stage 0 ..
    // STAGES-1], rows of BK bf16 (CPR 16-byte chunks, XOR-swizzled).  Wave
    // instruction q of a tile moves 64 lanes x 16 bytes = RPI tile rows; lane l
    // fills slot l % CPR of row l / CPR and so fetches the logical chunk that
    // the swizzle puts in that slot.  Loads are range-checked buffer loads
    // over the whole operand: rows past M / N read as zeros (their products
    // only reach discarded outputs).
    //
    // Every address is fixed before the loop: a lane's global offset of each
    // load instruction (the k offset of a tile travels in the scalar offset),
    // the LDS destination of each instruction (scalar, wave-uniform) and the
    // lane's LDS fragment address for each k-step (the stage and fragment
    // index are immediate offsets), so the loop issues MFMAs, LDS reads and
    // buffer loads and almost no vector ALU work.
    constexpr int RPI = 64 / CPR;                       // tile rows per instruction
    constexpr int AI = BM / RPI / NWAVES, BI = BN / RPI / NWAVES;
    static_assert(AI * RPI * NWAVES == BM && BI * RPI * NWAVES == BN, "tile config");
    constexpr int IPT = AI + BI;                        // load instructions per tile per wave
    constexpr int KS = BK / 16;                         // k-steps per tile
    constexpr int ROWB = CPR * 16;                      // bytes per LDS row
    constexpr int A_STAGE = BM * ROWB, B_STAGE = BN * ROWB;
    constexpr int B_REGION = STAGES * A_STAGE;
    static_assert(B_REGION + STAGES * B_STAGE <= (int)sizeof(lds), "LDS");
    static_assert((STAGES - 1) * A_STAGE + (FM - 1) * 32 * ROWB < 65536 &&
                  (STAGES - 1) * B_STAGE + (FN - 1) * 32 * ROWB < 65536, "ds_read immediate offsets");
    const int wv = __builtin_amdgcn_readfirstlane(wave);  // wave index in a scalar register
    const __amdgpu_buffer_rsrc_t rsa = __builtin_amdgcn_make_buffer_rsrc((void*)A, (short)0, (int)((long)M * lda * 2),
                                                                         kBufferWord3);
    const __amdgpu_buffer_rsrc_t rsw = __builtin_amdgcn_make_buffer_rsrc((void*)W, (short)0, (int)((long)N * ldw * 2),
                                                                         kBufferWord3);
    // per-lane global byte offsets of the load instructions (k offset excluded)
    int goa[AI], gob[BI];
    {
      const int lr = lane / CPR, sl = lane % CPR;
#pragma unroll
      for (int q = 0; q < AI; ++q) {
        const int row = (wv * AI + q) * RPI + lr;
        const int kc = lds_slot<CPR>(row, sl) - row * CPR;  // the XOR is an involution
        goa[q] = ((m0 + row) * (int)lda + kc * 8) * 2;
      }
#pragma unroll
      for (int q = 0; q < BI; ++q) {
        const int row = (wv * BI + q) * RPI + lr;
        const int kc = lds_slot<CPR>(row, sl) - row * CPR;
        gob[q] = ((n0 + row) * (int)ldw + kc * 8) * 2;
      }
    }
    // per-lane LDS byte address of fragment 0 at k-step ks, stage 0.  Rows of
    // fragment i differ by 32 i, which leaves the swizzle term unchanged.
    int fra[KS], frb[KS];
    {
      const int ra = wm * WTM + (lane & 31), rb = wn * WTN + (lane & 31);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        fra[ks] = lds_slot<CPR>(ra, 2 * ks + (lane >> 5)) * 16;
        frb[ks] = B_REGION + lds_slot<CPR>(rb, 2 * ks + (lane >> 5)) * 16;
      }
    }
    char* const lbase = (char*)lds;
    // load instructions [q0, q1) of tile kt (A's first, then B's) into stage st
    auto load_part = [&](int st, int kt, int q0, int q1) __attribute__((always_inline)) {
      const int koff = kt * BK * 2;
#pragma unroll
      for (int q = 0; q < AI; ++q) {
        if (q < q0 || q >= q1) continue;
        // copied to a local first: the array element passed straight to the
        // builtin makes the host pass drop the kernel launch stub
        const int vo = goa[q];
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rsa, (__attribute__((address_space(3))) void*)(lbase + st * A_STAGE + (wv * AI + q) * RPI * ROWB), 16,
            vo, koff, 0, 0);
      }
#pragma unroll
      for (int q = 0; q < BI; ++q) {
        if (AI + q < q0 || AI + q >= q1) continue;
        const int vo = gob[q];
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rsw,
            (__attribute__((address_space(3))) void*)(lbase + B_REGION + st * B_STAGE + (wv * BI + q) * RPI * ROWB),
            16, vo, koff, 0, 0);
      }
    };
    auto read_frags = [&](auto stc, auto ksc, auto bufc) __attribute__((always_inline)) {
      constexpr int st = decltype(stc)::value, ks = decltype(ksc)::value, buf = decltype(bufc)::value;
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[buf][i] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(lbase + fra[ks] + st * A_STAGE + i * 32 * ROWB));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        fb[buf][j] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(lbase + frb[ks] + st * B_STAGE + j * 32 * ROWB));
    };
    auto mfma_step = [&](auto bufc) __attribute__((always_inline)) {
      constexpr int buf = decltype(bufc)::value;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[buf][i], fb[buf][j], acc[i][j], 0, 0, 0);
    };
    constexpr int NR = FM + FN, NM = FM * FN, NP = NR < NM ? NR : NM;
    using I0 = std::integral_constant<int, 0>;
    if constexpr (M16) {
    // ---- as below, with v_mfma_f32_16x16x32_bf16: two 32-wide k-steps per
    // K tile, each split into two phases by fragment row; fragments of tile X
    // are read in X-1's last phase (k-step 0) and X's first phase (k-step 1).
    static_assert(BK == 64 && STAGES == 2, "schedule for 64-wide K tiles");
    constexpr int FM2 = 2 * FM, FN2 = 2 * FN, NR2 = FM2 + FN2, NMP = FM * FN2;  // MFMAs per phase
    static_assert((STAGES - 1) * A_STAGE + (FM2 - 1) * 16 * ROWB < 65536 &&
                  (STAGES - 1) * B_STAGE + (FN2 - 1) * 16 * ROWB < 65536, "ds_read immediate offsets");
    int fa16[2], fb16[2];
    {
      const int ra = wm * WTM + (lane & 15), rb = wn * WTN + (lane & 15);
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        fa16[ks] = lds_slot<CPR>(ra, 4 * ks + (lane >> 4)) * 16;
        fb16[ks] = B_REGION + lds_slot<CPR>(rb, 4 * ks + (lane >> 4)) * 16;
      }
    }
    bf16x8_t ha[2][FM2], hb[2][FN2];
    auto rd16 = [&](auto stc, auto ksc) __attribute__((always_inline)) {
      constexpr int st = decltype(stc)::value, ks = decltype(ksc)::value;
#pragma unroll
      for (int i = 0; i < FM2; ++i)
        ha[ks][i] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(lbase + fa16[ks] + st * A_STAGE + i * 16 * ROWB));
#pragma unroll
      for (int j = 0; j < FN2; ++j)
        hb[ks][j] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(lbase + fb16[ks] + st * B_STAGE + j * 16 * ROWB));
    };
    auto mm16 = [&](auto ksc, auto hc) __attribute__((always_inline)) {
      constexpr int ks = decltype(ksc)::value, h = decltype(hc)::value;
#pragma unroll
      for (int i = h * FM; i < (h + 1) * FM; ++i)
#pragma unroll
        for (int j = 0; j < FN2; ++j)
          acc16[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ha[ks][i], hb[ks][j], acc16[i][j], 0, 0, 0);
    };
    auto weave16 = [&](auto rc, auto vc) __attribute__((always_inline)) {
      constexpr int R = decltype(rc)::value, V = decltype(vc)::value;
      static_for<NMP>([&](auto mc) {
        constexpr int m = decltype(mc)::value;
        constexpr int r = (m + 1) * R / NMP - m * R / NMP, v = (m + 1) * V / NMP - m * V / NMP;
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);
        if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, 0);
      });
    };
    constexpr int QH = IPT / 2;
    using J0 = std::integral_constant<int, 0>;
    using J1 = std::integral_constant<int, 1>;
    auto tile16 = [&](auto stc, int kt) __attribute__((always_inline)) {
      constexpr int st = decltype(stc)::value;
      using SN = std::integral_constant<int, st ^ 1>;
      rd16(stc, J1{});
      mm16(J0{}, J0{});
      weave16(std::integral_constant<int, NR2>{}, J0{});
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
      asm volatile("s_barrier" ::: "memory");
      load_part(st, min(kt + 2, KT - 1), 0, QH);
      mm16(J0{}, J1{});
      weave16(J0{}, std::integral_constant<int, QH>{});
      __builtin_amdgcn_sched_barrier(0);
      load_part(st, min(kt + 2, KT - 1), QH, IPT);
      mm16(J1{}, J0{});
      weave16(J0{}, std::integral_constant<int, IPT - QH>{});
      __builtin_amdgcn_sched_barrier(0);
      wait_vmcnt<IPT>();
      asm volatile("s_barrier" ::: "memory");
      rd16(SN{}, J0{});
      mm16(J1{}, J1{});
      weave16(std::integral_constant<int, NR2>{}, J0{});
      __builtin_amdgcn_sched_barrier(0);
    };
    load_part(0, 0, 0, IPT);
    load_part(1, min(1, KT - 1), 0, IPT);
    wait_vmcnt<IPT>();
    asm volatile("s_barrier" ::: "memory");
    rd16(I0{}, J0{});
    int kt = 0;
    for (; kt + 1 < KT; kt += 2) {
      tile16(I0{}, kt);
      tile16(std::integral_constant<int, 1>{}, kt + 1);
    }
    if (kt < KT) tile16(I0{}, kt);
    } else if constexpr (kSchedK == 1) {
    // ---- whole-tile register prefetch, two barriers per K tile.
    // Fragment registers hold one whole K tile (one buffer per k-step).  The
    // fragments of tile X are read during the last k-step of tile X-1 (k-steps
    // 0, 1) and the first k-step of X (k-steps 2, 3); after a barrier at the
    // start of X's second k-step nobody reads X's stage any more and the loads
    // of tile X+2 into it are issued over X's k-steps 1 and 2 (about the rate
    // the texture path drains them); a second barrier before X's last k-step
    // makes tile X+1 visible.  A load thus has about one K tile between its
    // issue and the barrier that needs it.
    static_assert(KS == 4 && STAGES == 2, "schedule for 64-wide K tiles");
    bf16x8_t ga[KS][FM], gb[KS][FN];
    auto rd = [&](auto stc, auto ksc) __attribute__((always_inline)) {
      constexpr int st = decltype(stc)::value, ks = decltype(ksc)::value;
#pragma unroll
      for (int i = 0; i < FM; ++i)
        ga[ks][i] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(lbase + fra[ks] + st * A_STAGE + i * 32 * ROWB));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        gb[ks][j] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(lbase + frb[ks] + st * B_STAGE + j * 32 * ROWB));
    };
    auto mm = [&](auto ksc) __attribute__((always_inline)) {
      constexpr int ks = decltype(ksc)::value;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ga[ks][i], gb[ks][j], acc[i][j], 0, 0, 0);
    };
    // interleave: NM MFMAs with R DS reads and V VMEM loads spread evenly
    auto weave = [&](auto rc, auto vc) __attribute__((always_inline)) {
      constexpr int R = decltype(rc)::value, V = decltype(vc)::value;
      static_for<NM>([&](auto mc) {
        constexpr int m = decltype(mc)::value;
        constexpr int r = (m + 1) * R / NM - m * R / NM, v = (m + 1) * V / NM - m * V / NM;
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);
        if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, 0);
      });
    };
    // the loads of tile kt + 2 leave in NCH equal chunks: k-steps 1, 2 (and 3,
    // and the next tile's k-step 0) of tile kt
    constexpr int NCH = IPT % kLoadChunksK == 0 ? kLoadChunksK : 2;
    static_assert(NCH >= 2 && NCH <= 4 && IPT % NCH == 0, "load chunks");
    constexpr int QC = IPT / NCH;
    using K0 = std::integral_constant<int, 0>;
    using K1 = std::integral_constant<int, 1>;
    using K2 = std::integral_constant<int, 2>;
    using K3 = std::integral_constant<int, 3>;
    using RR = std::integral_constant<int, 2 * NR>;   // fragment reads of two k-steps
    using VQ = std::integral_constant<int, QC>;
    auto tile2 = [&](auto stc, int kt) __attribute__((always_inline)) {
      constexpr int st = decltype(stc)::value;
      using SN = std::integral_constant<int, st ^ 1>;
      // k-step 0: read this tile's k-steps 2, 3 (and the last chunk of tile kt + 1)
      rd(stc, K2{});
      rd(stc, K3{});
      if constexpr (NCH == 4) load_part(st ^ 1, min(kt + 1, KT - 1), 3 * QC, IPT);
      mm(K0{});
      weave(RR{}, std::integral_constant<int, NCH == 4 ? QC : 0>{});
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): own reads of this stage done
      asm volatile("s_barrier" ::: "memory");
      // k-steps 1, 2: loads of tile kt + 2 into this stage
      load_part(st, min(kt + 2, KT - 1), 0, QC);
      mm(K1{});
      weave(K0{}, VQ{});
      __builtin_amdgcn_sched_barrier(0);
      load_part(st, min(kt + 2, KT - 1), QC, 2 * QC);
      mm(K2{});
      weave(K0{}, VQ{});
      __builtin_amdgcn_sched_barrier(0);
      // tile kt + 1 landed (the chunks of kt + 2 issued so far may still be in flight)
      wait_vmcnt<2 * QC>();
      asm volatile("s_barrier" ::: "memory");
      // k-step 3: read the next tile's k-steps 0, 1
      rd(SN{}, K0{});
      rd(SN{}, K1{});
      if constexpr (NCH >= 3) load_part(st, min(kt + 2, KT - 1), 2 * QC, 3 * QC);
      mm(K3{});
      weave(RR{}, std::integral_constant<int, NCH >= 3 ? QC : 0>{});
      __builtin_amdgcn_sched_barrier(0);
    };
    load_part(0, 0, 0, IPT);
    load_part(1, min(1, KT - 1), 0, NCH == 4 ? 3 * QC : IPT);
    wait_vmcnt<NCH == 4 ? 3 * QC : IPT>();
    asm volatile("s_barrier" ::: "memory");
    rd(I0{}, K0{});
    rd(I0{}, K1{});
    int kt = 0;
    for (; kt + 1 < KT; kt += 2) {
      tile2(I0{}, kt);
      tile2(std::integral_constant<int, 1>{}, kt + 1);
    }
    if (kt < KT) tile2(I0{}, kt);
    } else {
    // One K tile in stage st: k-steps 0 .. KS-2 (each k-step's MFMAs alternate
    // with the fragment reads of the next), then the barrier before the last
    // k-step: after it this stage is free, and the first fragments of the next
    // tile are read under the last k-step's MFMAs, so no wave idles between
    // tiles.  The loads of tile kt + 2 into this stage are spread over LSPLIT
    // k-steps -- the last one of this tile and the first LSPLIT - 1 of the
    // next -- instead of leaving in one burst.  Loads past the last K tile
    // fetch it again into a buffer nobody reads any more (no branches,
    // constant wait counts).  The barrier is a bare s_barrier: a
    // __syncthreads() fence would also drain the loads still in flight.
    constexpr int LSPLIT = IPT % kLoadSplitK == 0 ? kLoadSplitK : 1;
    static_assert(LSPLIT >= 1 && LSPLIT <= KS && IPT % LSPLIT == 0, "load split");
    constexpr int QC = IPT / LSPLIT;  // load instructions per chunk
    auto tile = [&](auto stc, int kt) __attribute__((always_inline)) {
      constexpr int st = decltype(stc)::value;
      static_for<KS - 1>([&](auto kk) {
        constexpr int ks = decltype(kk)::value;
        read_frags(stc, std::integral_constant<int, ks + 1>{}, std::integral_constant<int, (ks + 1) & 1>{});
        constexpr bool ld = ks + 1 < LSPLIT;
        if constexpr (ld) load_part(st ^ 1, min(kt + 1, KT - 1), (ks + 1) * QC, (ks + 2) * QC);
        mfma_step(std::integral_constant<int, ks & 1>{});
        constexpr int VP = ld ? (QC / NP > 0 ? QC / NP : 1) : 0;
        static_for<NP>([&](auto) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          if constexpr (VP > 0) __builtin_amdgcn_sched_group_barrier(0x020, VP, 0);  // VMEM
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
        });
        if constexpr (NM > NP) __builtin_amdgcn_sched_group_barrier(0x008, NM - NP, 0);
        if constexpr (NR > NP) __builtin_amdgcn_sched_group_barrier(0x100, NR - NP, 0);
      });
      // own loads of tile kt + 1 done and the last fragments of tile kt read;
      // after the barrier tile kt + 1 is in LDS and nobody reads stage st
      wait_vmcnt<0>();
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
      asm volatile("s_barrier" ::: "memory");
      load_part(st, min(kt + 2, KT - 1), 0, QC);
      read_frags(std::integral_constant<int, st ^ 1>{}, I0{}, I0{});
      mfma_step(std::integral_constant<int, (KS - 1) & 1>{});
      constexpr int VP = QC / NP > 0 ? QC / NP : 1;
      static_for<NP>([&](auto) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
        __builtin_amdgcn_sched_group_barrier(0x020, VP, 0);  // VMEM (buffer -> LDS)
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
      });
    };
    static_assert(STAGES == 2, "the unrolled loop alternates two stages");
    using I1 = std::integral_constant<int, 1>;
    load_part(0, 0, 0, IPT);
    load_part(1, min(1, KT - 1), 0, QC);
    wait_vmcnt<QC>();
    asm volatile("s_barrier" ::: "memory");
    read_frags(I0{}, I0{}, I0{});
    int kt = 0;
    for (; kt + 1 < KT; kt += 2) {
      tile(I0{}, kt);
      tile(I1{}, kt + 1);
    }
    if (kt < KT) tile(I0{}, kt);
    }
    // the refetches of the last tile must land before the epilogue reuses LDS
    wait_vmcnt<0>();
    __syncthreads();
  } else {
    // ---- register path with zero-filled K tail (two LDS buffers).
    constexpr int A_CH = BM * CPR / NT, B_CH = BN * CPR / NT;
    static_assert((BM * CPR) % NT == 0 && (BN * CPR) % NT == 0 && A_CH >= 1 && B_CH >= 1, "tile config");
    uint4 ra[A_CH], rb[B_CH];
    auto gload = [&](int kt) {
      const int k0 = kt * BK;
#pragma unroll
      for (int c = 0; c < A_CH; ++c) {
        const int idx = tid + c * NT;
        const int row = idx / CPR, kc = idx % CPR;
        const int gr = m0 + row, gk = k0 + kc * 8;
        const bool ok = gr < M && gk < K;
        const uint4 v = *(const uint4*)(A + (long)min(gr, M - 1) * lda + min(gk, K - 8));
        ra[c] = ok ? v : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int c = 0; c < B_CH; ++c) {
        const int idx = tid + c * NT;
        const int row = idx / CPR, kc = idx % CPR;
        const int gr = n0 + row, gk = k0 + kc * 8;
        const bool ok = gr < N && gk < K;
        const uint4 v = *(const uint4*)(W + (long)min(gr, N - 1) * ldw + min(gk, K - 8));
        rb[c] = ok ? v : make_uint4(0, 0, 0, 0);
      }
    };
    auto lstore = [&](int st) {
      uint4* S = lds + st * STAGE;
#pragma unroll
      for (int c = 0; c < A_CH; ++c) {
        const int idx = tid + c * NT;
        S[lds_slot<CPR>(idx / CPR, idx % CPR)] = ra[c];
      }
#pragma unroll
      for (int c = 0; c < B_CH; ++c) {
        const int idx = tid + c * NT;
        S[lds_slot<CPR>(BM + idx / CPR, idx % CPR)] = rb[c];
      }
    };
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      if (kt + 1 < KT) gload(kt + 1);
      compute(kt & 1);
      if (kt + 1 < KT) lstore((kt + 1) & 1);
      __syncthreads();
    }
  }

  // epilogue.  Row facts (request, joint position, grid position) are computed
  // once per tile row into LDS, so the unrolled loops never index the batch
  // metadata.  Each 32x32 accumulator fragment is staged through a per-wave
  // LDS buffer so that a lane ends up with 16 consecutive columns of one row
  // and stores them with 16-byte writes.
  RowEntry* rows = (RowEntry*)&lds[0];
  constexpr int SP = 36;  // staging row pitch in floats (16-byte aligned rows)
  float* stg = (float*)&lds[0] + BM * (sizeof(RowEntry) / 4) + wave * 32 * SP;
  static_assert(BM * sizeof(RowEntry) + NWAVES * 32 * SP * 4 <= sizeof(lds), "epilogue LDS");
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
    // V^T columns of a QKV epilogue: a lane takes one column and 16 consecutive
    // rows, which (when they are 16 consecutive, 16-aligned joint positions of
    // one request) land in one aligned 16-key group of V^T: two 16-byte stores.
    const bool vcols = E.mode == EPI_QKV && nb >= 2 * E.hidden && nb < 3 * E.hidden;
    static_for<FM>([&](auto ii) {
      constexpr int i = decltype(ii)::value;
      if constexpr (M16) {
        static_for<2>([&](auto bb) {
          constexpr int b = decltype(bb)::value;
          const int nl16 = nb + b * 16 + (lane & 15);
          const float bn16 = (bias != nullptr && nl16 < N) ? bf2f(bias[nl16]) : 0.f;
          static_for<2>([&](auto aa) {
            constexpr int a = decltype(aa)::value;
            static_for<4>([&](auto rr) {
              constexpr int r = decltype(rr)::value;
              stg[(a * 16 + 4 * (lane >> 4) + r) * SP + b * 16 + (lane & 15)] = acc16[2 * i + a][2 * j + b][r] + bn16;
            });
          });
        });
      } else {
        static_for<16>([&](auto rr) {
          constexpr int r = decltype(rr)::value;
          stg[((r / 4) * 8 + (lane >> 5) * 4 + (r % 4)) * SP + (lane & 31)] = acc[i][j][r] + bn;
        });
      }
      if (vcols) {
        const int rh = lane >> 5, c = lane & 31;
        float v[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) v[q] = stg[(rh * 16 + q) * SP + c];
        const int ml0 = wm * WTM + i * 32 + rh * 16;
        const int m = m0 + ml0, n = nb + c;
        if (n < N && m < M) {
          const RowEntry r0 = rows[ml0];
          const bool whole = m + 15 < M && (r0.pos & 15) == 0 && rows[ml0 + 15].pos == r0.pos + 15;
          const int hn = n - 2 * E.hidden, h = hn / E.head_dim, dd = hn - h * E.head_dim;
          bf16_t* vt = (bf16_t*)E.vt + ((long)h * E.head_dim + dd) * E.T;
          if (whole) {
            // slot s of the group holds key vt_slot(s): swap the middle quads
            float w[16];
#pragma unroll
            for (int q = 0; q < 16; ++q) w[q] = v[vt_slot(q)];
            store16<bf16_t>(vt + r0.pos, w);
          } else {
#pragma unroll
            for (int q = 0; q < 16; ++q)
              if (m + q < M) vt[vt_slot(rows[ml0 + q].pos)] = f2bf(v[q]);
          }
        }
        return;
      }
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

// direct-to-LDS path: whole K tiles, 16-byte aligned rows, and operands
// small enough for the 32-bit offsets of buffer loads
template <int BM, int BN, int BK>
bool dtl_ok(const GemmProblem& p) {
  for (int g = 0; g < p.n_groups; ++g) {
    const GemmGroup& G = p.g[g];
    const bool ok = G.K % BK == 0 && G.lda % 8 == 0 && G.ldw % 8 == 0 && (long)(G.M + BM) * G.lda * 2 < (1L << 31) &&
                    (long)(p.N + BN) * G.ldw * 2 < (1L << 31);
    if (!ok) return false;
  }
  return true;
}

template <int BM, int BN>
long tile_count(const GemmProblem& p) {
  const int tiles_n = (p.N + BN - 1) / BN;
  long tiles = (long)((p.g[0].M + BM - 1) / BM) * tiles_n;
  if (p.n_groups > 1) tiles += (long)((p.g[1].M + BM - 1) / BM) * tiles_n;
  return tiles;
}

template <int BM, int BN, int NWM, int NWN, int BK, int STAGES, bool DTL>
hipError_t launch_kernel(const GemmProblem& p, hipStream_t s) {
  const long tiles = tile_count<BM, BN>(p);
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, NWM, NWN, BK, STAGES, DTL>), dim3((unsigned)tiles),
                     dim3(NWM * NWN * 64), 0, s, p);
  return hipGetLastError();
}

template <int BM, int BN, int NWM, int NWN, int BK, int STAGES>
hipError_t launch_cfg(const GemmProblem& p, hipStream_t s) {
  if (dtl_ok<BM, BN, BK>(p)) return launch_kernel<BM, BN, NWM, NWN, BK, STAGES, true>(p, s);
  return launch_kernel<BM, BN, NWM, NWN, BK, STAGES, false>(p, s);
}

constexpr bool kWaves4 = false;

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
      return launch_cfg<128, 64, 4, 1, 64, 2>(p, s);
    case CFG_256x256:
      if (dtl_ok<256, 256, 64>(p))
        return kWaves4 ? launch_kernel<256, 256, 2, 2, 64, 2, true>(p, s)
                       : launch_kernel<256, 256, 4, 2, 64, 2, true>(p, s);
      return launch_kernel<256, 256, 4, 2, 64, 2, false>(p, s);
    default:
      return launch_cfg<128, 128, 2, 2, 64, 2>(p, s);
  }
}

}  // namespace dit
