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
#include <string>

#include "device_common.h"

namespace dit {

namespace {


struct TileCoord {
  int group, m0, n0;
};

template <int BM, int BN>
__device__ __forceinline__ TileCoord tile_coord(const GemmProblem& P, int id) {
  const int tiles_n = (P.N + BN - 1) / BN;
  const int tm0 = (P.g[0].M + BM - 1) / BM;
  const int tiles0 = tm0 * tiles_n;
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

template <int n>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(n >= 0 && n < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef int i32x4_t __attribute__((ext_vector_type(4)));

// Single instructions as volatile asm statements, which the compiler keeps in
// the order written: a main loop built from them runs exactly its schedule.
// The compiler does not see what they do, so the loop that uses them issues
// its own LDS waits, and wait states separate its last MFMAs from any other
// reader of the accumulators.
template <int OFF>
__device__ __forceinline__ void asm_lds_read16(i32x4_t& d, int addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(d) : "v"(addr), "i"(OFF));
}
__device__ __forceinline__ void asm_mfma16(f32x4_t& c, const i32x4_t& a, const i32x4_t& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b));
}
// wait until at most N LDS operations of this wave are outstanding; none is
// emitted for N >= 15, since the counter never holds more than 15
template <int N>
__device__ __forceinline__ void asm_lgkm_wait() {
  if constexpr (N < 15) asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(N));
}

template <int BM, int BN, int NWM, int NWN, int BK, int STAGES, bool DTL>
__global__ __launch_bounds__(NWM* NWN * 64) void gemm_bf16_kernel(const GemmProblem P) {
  constexpr int NT = NWM * NWN * 64;
  constexpr int NWAVES = NWM * NWN;
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  // wave tiles: rows in 32-row fragments; columns in 32-column fragments on
  // the register path, in 16-column fragments on the direct-to-LDS path
  constexpr int FM = WTM / 32, FN = WTN / 32, FN16 = WTN / 16;
  constexpr int CPR = BK / 8;                     // 16-byte chunks per tile row
  constexpr int STAGE = (BM + BN) * CPR;          // uint4 per stage
  static_assert(FM * 32 == WTM && FN16 * 16 == WTN && (DTL || FN * 32 == WTN), "wave tile");
  static_assert(FM >= 1 && FN16 >= 1 && (BK == 32 || BK == 64) && STAGES >= 2 && BK % 32 == 0, "tile config");
  static_assert(STAGES * STAGE * 16 <= 160 * 1024, "LDS");

  __shared__ uint4 lds[STAGES * STAGE];

  // tile of this block and, when K is split, its piece; the pieces of a tile
  // have consecutive indices and so run on one XCD
  int tile_id = xcd_remap(blockIdx.x, gridDim.x), piece = 0;
  const int np = DTL ? P.sk_p : 1;
  if (np > 1) {
    piece = tile_id % np;
    tile_id /= np;
  }
  const TileCoord tc = tile_coord<BM, BN>(P, tile_id);
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

  // Accumulators.  Direct-to-LDS path: 16x16 blocks, the 32x32 fragment
  // (i, j) being the 2 x 2 blocks 2i.., 2j..; register path: 32x32 blocks.
  constexpr int AM = DTL ? 2 * FM : 1, AN = DTL ? FN16 : 1;
  constexpr int CM = DTL ? 1 : FM, CN = DTL ? 1 : FN;
  f32x4_t acc16[AM][AN];
  f32x16_t acc[CM][CN];
#pragma unroll
  for (int i = 0; i < AM; ++i)
#pragma unroll
    for (int j = 0; j < AN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc16[i][j][r] = 0.f;
#pragma unroll
  for (int i = 0; i < CM; ++i)
#pragma unroll
    for (int j = 0; j < CN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // K tiles [kb, kb + KT) of this block
  const int KT_all = (K + BK - 1) / BK;
  const int kb = piece * KT_all / np;
  const int KT = (piece + 1) * KT_all / np - kb;

  // register path: fragments of k-step ks (16 wide) of stage st: lane row
  // (lane & 31), chunk 2 ks + lane / 32
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
    // ---- direct-to-LDS ring.  LDS holds [A stage 0 | A stage 1 | B stage 0 |
    // B stage 1], rows of BK bf16 (CPR 16-byte chunks, XOR-swizzled).  Wave
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
    // buffer loads and no vector ALU work.
    //
    // MFMAs are v_mfma_f32_16x16x32_bf16: a 64-wide K tile is two 32-wide
    // k-steps, each split into two phases by fragment row, four phases of
    // FM x 2FN MFMAs.  Fragment registers hold one whole K tile.  Tile X is
    // read in the last phase of X-1 (k-step 0) and the first phase of X
    // (k-step 1); a barrier after X's first phase frees X's stage and the
    // loads of tile X+2 into it are spread over phases 1 and 2; a second
    // barrier, in the last phase ahead of its fragment reads, makes tile X+1
    // visible.  A load thus has about one K tile between its issue and the
    // barrier that needs it.
    static_assert(BK == 64 && STAGES == 2, "schedule for 64-wide K tiles, two stages");
    constexpr int RPI = 64 / CPR;                       // tile rows per instruction
    constexpr int AI = BM / RPI / NWAVES, BI = BN / RPI / NWAVES;
    static_assert(AI * RPI * NWAVES == BM && BI * RPI * NWAVES == BN, "tile config");
    constexpr int IPT = AI + BI;                        // load instructions per tile per wave
    constexpr int ROWB = CPR * 16;                      // bytes per LDS row
    constexpr int A_STAGE = BM * ROWB, B_STAGE = BN * ROWB;
    constexpr int B_REGION = STAGES * A_STAGE;
    constexpr int FM2 = 2 * FM, FN2 = FN16;             // 16-row / 16-column fragments per wave tile
    constexpr int NR2 = FM2 + FN2;                      // fragment reads per k-step
    constexpr int NMP = FM * FN2;                       // MFMAs per phase
    static_assert(B_REGION + STAGES * B_STAGE <= (int)sizeof(lds), "LDS");
    static_assert((STAGES - 1) * A_STAGE + (FM2 - 1) * 16 * ROWB < 65536 &&
                  (STAGES - 1) * B_STAGE + (FN2 - 1) * 16 * ROWB < 65536, "ds_read immediate offsets");
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
    // per-lane LDS byte address of fragment 0 at k-step ks, stage 0: row
    // lane % 16, chunk 4 ks + lane / 16.  Rows of fragment i differ by 16 i,
    // which leaves the swizzle term unchanged.
    int fra[2], frb[2];
    {
      const int ra = wm * WTM + (lane & 15), rb = wn * WTN + (lane & 15);
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        fra[ks] = lds_slot<CPR>(ra, 4 * ks + (lane >> 4)) * 16;
        frb[ks] = B_REGION + lds_slot<CPR>(rb, 4 * ks + (lane >> 4)) * 16;
      }
    }
    char* const lbase = (char*)lds;
    // load instructions [q0, q1) of tile kt (A's first, then B's) into stage st
    auto load_part = [&](int st, int kt, int q0, int q1) __attribute__((always_inline)) {
      const int koff = (kb + kt) * BK * 2;
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
    if constexpr (FM2 + FN2 <= FM * FN2) {
      // Every configuration whose phase holds at least one MFMA per fragment
      // read (all but the 128x64 skinny tile): the schedule below with every
      // MFMA, fragment read, LDS wait and barrier an asm statement, so the
      // instructions issue in exactly this order (0.5-2.5% faster than the
      // compiler's placement of the same schedule, bitwise the same results).
      // Phases of NMP MFMAs:
      //  P0  k-step 0, fragment rows 0 .. NA/2-1; one read of this tile's
      //      k-step-1 fragments after each of the first NR MFMAs
      //      -- lgkmcnt(0), barrier: no wave reads this stage any more
      //  P1  k-step 0, rows NA/2 ..; loads 0 .. Q1-1 of tile kt+2 spread over it
      //  P2  k-step 1, rows 0 .. NA/2-1; the other IPT - Q1 loads
      //  P3  k-step 1, rows NA/2 ..: NMP - NR MFMAs, then
      //      -- vmcnt(IPT), barrier: tile kt+1 visible
      //      the rest, each followed by one of the next tile's k-step-0 reads
      // LDS operations complete in order, so before each P0 MFMA the wait
      // allows every read issued after the P3 read that MFMA needs.
      constexpr int NA = FM2, NB = FN2, NR = NA + NB, NMP = (NA / 2) * NB;
      static_assert(NR <= NMP, "schedule");
      const int lds0 = (int)(unsigned)(size_t)(__attribute__((address_space(3))) char*)lbase;
      const int a0 = lds0 + fra[0], a1 = lds0 + fra[1], b0 = lds0 + frb[0], b1 = lds0 + frb[1];
      i32x4_t fa0[NA], fb0[NB], fa1[NA], fb1[NB];
      // k-step-0 fragment reads in the order A0, B0 .. B(NB-1), A1 .. A(NA-1)
      // (the order the first P0 MFMAs need them); k-step 1: A's, then B's
      auto rd0 = [&](auto stc, auto rc) __attribute__((always_inline)) {
        constexpr int st = decltype(stc)::value, r = decltype(rc)::value;
        if constexpr (r == 0) asm_lds_read16<st * A_STAGE>(fa0[0], a0);
        else if constexpr (r <= NB) asm_lds_read16<st * B_STAGE + (r - 1) * 16 * ROWB>(fb0[r - 1], b0);
        else asm_lds_read16<st * A_STAGE + (r - NB) * 16 * ROWB>(fa0[r - NB], a0);
      };
      auto rd1 = [&](auto stc, auto rc) __attribute__((always_inline)) {
        constexpr int st = decltype(stc)::value, r = decltype(rc)::value;
        if constexpr (r < NA) asm_lds_read16<st * A_STAGE + r * 16 * ROWB>(fa1[r], a1);
        else asm_lds_read16<st * B_STAGE + (r - NA) * 16 * ROWB>(fb1[r - NA], b1);
      };
      // loads [Q1) of a tile in P1 and [Q1, IPT) in P2, spread evenly over each phase's MFMAs
      constexpr int Q1 = (IPT + 1) / 2, Q2 = IPT - Q1;
      auto tile8 = [&](auto stc, int kt) __attribute__((always_inline)) {
        constexpr int st = decltype(stc)::value;
        using SN = std::integral_constant<int, st ^ 1>;
        const int kt2 = min(kt + 2, KT - 1);
        static_for<NMP>([&](auto mc) {  // P0: k-step 0, rows 0 .. NA/2-1; this tile's k-step-1 reads
          constexpr int m = decltype(mc)::value, i = m / NB, j = m % NB;
          constexpr int ia = i == 0 ? 0 : NB + i, ib = 1 + j;
          constexpr int need = ia > ib ? ia : ib;
          asm_lgkm_wait<(NR - 1 - need) + (m < NR ? m : NR)>();
          asm_mfma16(acc16[i][j], fa0[i], fb0[j]);
          if constexpr (m < NR) rd1(stc, std::integral_constant<int, m>{});
        });
        asm_lgkm_wait<0>();
        asm volatile("s_barrier" ::: "memory");
        static_for<NMP>([&](auto mc) {  // P1: k-step 0, rows NA/2 ..; first half of the loads of tile kt+2
          constexpr int m = decltype(mc)::value, i = NA / 2 + m / NB, j = m % NB;
          asm_mfma16(acc16[i][j], fa0[i], fb0[j]);
          constexpr int q0 = m * Q1 / NMP, q1 = (m + 1) * Q1 / NMP;
          if constexpr (q1 > q0) load_part(st, kt2, q0, q1);
        });
        static_for<NMP>([&](auto mc) {  // P2: k-step 1, rows 0 .. NA/2-1; second half of the loads
          constexpr int m = decltype(mc)::value, i = m / NB, j = m % NB;
          asm_mfma16(acc16[i][j], fa1[i], fb1[j]);
          constexpr int q0 = m * Q2 / NMP, q1 = (m + 1) * Q2 / NMP;
          if constexpr (q1 > q0) load_part(st, kt2, Q1 + q0, Q1 + q1);
        });
        static_for<NMP>([&](auto mc) {  // P3: k-step 1, rows NA/2 ..; the next tile's k-step-0 reads
          constexpr int m = decltype(mc)::value, i = NA / 2 + m / NB, j = m % NB;
          if constexpr (m == NMP - NR) {  // the MFMAs before it need no LDS
            wait_vmcnt<IPT>();
            asm volatile("s_barrier" ::: "memory");
          }
          asm_mfma16(acc16[i][j], fa1[i], fb1[j]);
          if constexpr (m >= NMP - NR) rd0(SN{}, std::integral_constant<int, m - (NMP - NR)>{});
        });
      };
      // The zeroed accumulators pass through an empty asm statement here, so
      // their initialisation is issued before the prologue and not next to
      // the first asm MFMA (a VALU write just before an MFMA that reads it
      // needs wait states the compiler does not know to insert).
#pragma unroll
      for (int i = 0; i < NA; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) asm volatile("" : "+v"(acc16[i][j]));
      load_part(0, 0, 0, IPT);
      load_part(1, min(1, KT - 1), 0, IPT);
      wait_vmcnt<IPT>();
      asm volatile("s_barrier" ::: "memory");
      static_for<NR>([&](auto rc) { rd0(std::integral_constant<int, 0>{}, rc); });
      int kt = 0;
      for (; kt + 1 < KT; kt += 2) {
        tile8(std::integral_constant<int, 0>{}, kt);
        tile8(std::integral_constant<int, 1>{}, kt + 1);
      }
      if (kt < KT) tile8(std::integral_constant<int, 0>{}, kt);
      asm_lgkm_wait<0>();
      // wait states between the last asm MFMAs and the accumulators' next
      // reader; each accumulator then passes through an empty asm statement,
      // which keeps every read of it after the wait states
      asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
      for (int i = 0; i < NA; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) asm volatile("" : "+v"(acc16[i][j]));
    } else {
    bf16x8_t ha[2][FM2], hb[2][FN2];
      auto rd = [&](auto stc, auto ksc) __attribute__((always_inline)) {
        constexpr int st = decltype(stc)::value, ks = decltype(ksc)::value;
  #pragma unroll
        for (int i = 0; i < FM2; ++i)
          ha[ks][i] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(lbase + fra[ks] + st * A_STAGE + i * 16 * ROWB));
  #pragma unroll
        for (int j = 0; j < FN2; ++j)
          hb[ks][j] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(lbase + frb[ks] + st * B_STAGE + j * 16 * ROWB));
      };
      // phase h of k-step ks: fragment rows h FM .. (h + 1) FM - 1
      auto mm = [&](auto ksc, auto hc) __attribute__((always_inline)) {
        constexpr int ks = decltype(ksc)::value, h = decltype(hc)::value;
  #pragma unroll
        for (int i = h * FM; i < (h + 1) * FM; ++i)
  #pragma unroll
          for (int j = 0; j < FN2; ++j)
            acc16[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ha[ks][i], hb[ks][j], acc16[i][j], 0, 0, 0);
      };
      // instruction order of a phase: each MFMA followed by its share of R LDS
      // reads and V buffer loads
      auto weave = [&](auto rc, auto vc) __attribute__((always_inline)) {
        constexpr int R = decltype(rc)::value, V = decltype(vc)::value;
        static_for<NMP>([&](auto mc) {
          constexpr int m = decltype(mc)::value;
          constexpr int r = (m + 1) * R / NMP - m * R / NMP, v = (m + 1) * V / NMP - m * V / NMP;
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                           // MFMA
          if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);      // DS read
          if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, 0);      // VMEM read
        });
      };
      constexpr int QH = IPT / 2;
      using J0 = std::integral_constant<int, 0>;
      using J1 = std::integral_constant<int, 1>;
      auto tile = [&](auto stc, int kt) __attribute__((always_inline)) {
        constexpr int st = decltype(stc)::value;
        using SN = std::integral_constant<int, st ^ 1>;
        // phase 0: this tile's k-step 1 fragments
        rd(stc, J1{});
        mm(J0{}, J0{});
        weave(std::integral_constant<int, NR2>{}, J0{});
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): own reads of this stage done
        asm volatile("s_barrier" ::: "memory");
        // phases 1, 2: the loads of tile kt + 2 into this stage
        load_part(st, min(kt + 2, KT - 1), 0, QH);
        mm(J0{}, J1{});
        weave(J0{}, std::integral_constant<int, QH>{});
        __builtin_amdgcn_sched_barrier(0);
        load_part(st, min(kt + 2, KT - 1), QH, IPT);
        mm(J1{}, J0{});
        weave(J0{}, std::integral_constant<int, IPT - QH>{});
        __builtin_amdgcn_sched_barrier(0);
        // tile kt + 1 landed (only the loads of kt + 2 may still be in flight)
        wait_vmcnt<IPT>();
        asm volatile("s_barrier" ::: "memory");
        // phase 3: the next tile's k-step 0 fragments
        rd(SN{}, J0{});
        mm(J1{}, J1{});
        weave(std::integral_constant<int, NR2>{}, J0{});
        __builtin_amdgcn_sched_barrier(0);
      };
      // Loads past the last K tile fetch it again into a stage nobody reads any
      // more (no branches, constant wait counts).  The barriers are bare
      // s_barriers: a __syncthreads() fence would also drain the loads still in
      // flight for later tiles.
      load_part(0, 0, 0, IPT);
      load_part(1, min(1, KT - 1), 0, IPT);
      wait_vmcnt<IPT>();
      asm volatile("s_barrier" ::: "memory");
      rd(J0{}, J0{});
      int kt = 0;
      for (; kt + 1 < KT; kt += 2) {
        tile(J0{}, kt);
        tile(J1{}, kt + 1);
      }
      if (kt < KT) tile(J0{}, kt);
    }
    // the refetches of the last tile must land before the epilogue reuses LDS
    wait_vmcnt<0>();
    __syncthreads();

    if (np > 1) {
      // Split K: publish this piece's partial sums, or -- for the last piece
      // of the tile to arrive -- add every piece's in piece order (the same
      // order whichever piece arrives last) and go on to the epilogue.  A
      // piece that finds all the others already counted skips publishing.
      // Only thread 0 orders memory: every wave waits for its own stores
      // before the block barrier, thread 0 then releases at agent scope
      // (writing the XCD's L2 back) and counts, and only a block that reads
      // the others' sums acquires (an acquire invalidates the L2 of its XCD,
      // which blocks still multiplying there depend on).
      constexpr int NV = AM * AN;
      int* const flag = (int*)&lds[STAGES * STAGE - 1];  // past the epilogue's LDS (asserted below)
      int* const cnt = P.sk_cnt + tile_id;
      float4* const slots = (float4*)P.sk_part + (long)tile_id * np * NV * NT;
      if (tid == 0) {
        const bool last = __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == np - 1;
        if (last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        *flag = last;
      }
      __syncthreads();
      if (!*flag) {
        float4* const mine = slots + (long)piece * NV * NT;
#pragma unroll
        for (int i = 0; i < AM; ++i)
#pragma unroll
          for (int j = 0; j < AN; ++j) {
            const f32x4_t a4 = acc16[i][j];
            mine[(i * AN + j) * NT + tid] = make_float4(a4[0], a4[1], a4[2], a4[3]);
          }
        // every wave's partial sums reach L2 before the barrier: the block
        // barrier alone does not wait for other waves' stores, and thread 0's
        // release below only waits for its own wave's
        wait_vmcnt<0>();
        __syncthreads();
        if (tid == 0) {
          // release: the XCD's L2 written back, and the write-back complete,
          // before the count
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
          wait_vmcnt<0>();
          const bool last = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == np - 1;
          if (last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
          *flag = last;
        }
        __syncthreads();
        if (!*flag) return;  // uniform across the block
      }
#pragma unroll
      for (int i = 0; i < AM; ++i)
#pragma unroll
        for (int j = 0; j < AN; ++j) {
          f32x4_t t = {0.f, 0.f, 0.f, 0.f};
          for (int qq = 0; qq < np; ++qq) {
            if (qq == piece) {
              t += acc16[i][j];
            } else {
              const float4 v = slots[((long)qq * NV + i * AN + j) * NT + tid];
              t[0] += v.x;
              t[1] += v.y;
              t[2] += v.z;
              t[3] += v.w;
            }
          }
          acc16[i][j] = t;
        }
      if (tid == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
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

  // epilogue.  Row facts (request, padded position, grid position) are computed
  // once per tile row into LDS, so the unrolled loops never index the batch
  // metadata.  Each 32x32 accumulator fragment is staged through a per-wave
  // LDS buffer so that a lane ends up with 16 consecutive columns of one row
  // and stores them with 16-byte writes.
  RowEntry* rows = (RowEntry*)&lds[0];
  constexpr int SP = 36;  // staging row pitch in floats (16-byte aligned rows)
  float* stg = (float*)&lds[0] + BM * (sizeof(RowEntry) / 4) + wave * 32 * SP;
  static_assert(BM * sizeof(RowEntry) + NWAVES * 32 * SP * 4 <= sizeof(lds) - 16, "epilogue LDS (the last 16 bytes hold the split flag)");
  const EpiArgs E = gi ? P.g[1].epi : P.g[0].epi;
  const bool need_rows = E.mode == EPI_RESID || E.mode == EPI_QKV;
  if (need_rows) {
    for (int t = tid; t < BM; t += NT)
      if (m0 + t < M) rows[t] = make_row_entry(P.meta, E.row_base + m0 + t);
    __syncthreads();
  }
  const bf16_t* bias = (const bf16_t*)E.bias;
  // The bias of every column this lane stages, loaded before the first output
  // store: loads and stores share one in-order counter, so a bias load issued
  // after a column group's stores would wait for them, and the groups would
  // follow one another at the latency of their stores.
  constexpr int NBC = DTL ? FN16 : FN;
  float bcol[NBC];
#pragma unroll
  for (int q = 0; q < NBC; ++q) {
    const int n = n0 + wn * WTN + (DTL ? q * 16 + (lane & 15) : q * 32 + (lane & 31));
    bcol[q] = (bias != nullptr && n < N) ? bf2f(bias[n]) : 0.f;
  }
  const int rl = lane >> 1, cseg = (lane & 1) * 16;
  // column groups of 32 (the last one 16 wide when the wave tile is an odd
  // number of 16-column fragments)
  constexpr int NJ = DTL ? (FN16 + 1) / 2 : FN;
  // Row groups outer, column groups inner: a lane's consecutive column groups
  // write adjacent pieces of the same rows (64 bytes of bf16 output each).
  static_for<FM>([&](auto ii) {
    constexpr int i = decltype(ii)::value;
    static_for<NJ>([&](auto jj) {
      constexpr int j = decltype(jj)::value;
      constexpr int NB16 = DTL ? (FN16 - 2 * j < 2 ? FN16 - 2 * j : 2) : 2;  // 16-column blocks in the group
      constexpr int NCOL = 16 * NB16;
      const int nb = n0 + wn * WTN + j * 32;
      const float bn = DTL ? 0.f : bcol[j];
      // V^T columns of a QKV epilogue: a lane takes one column and 16 consecutive
      // rows, which (when they are 16 consecutive, 16-aligned padded positions of
      // one request) land in one aligned 16-key group of V^T: two 16-byte stores.
      const bool vcols = E.mode == EPI_QKV && nb >= 2 * E.hidden && nb < 3 * E.hidden;
      if constexpr (DTL) {
        static_for<NB16>([&](auto bb) {
          constexpr int b = decltype(bb)::value;
          const float bn16 = bcol[2 * j + b];
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
        if (c < NCOL && n < N && m < M) {
          const RowEntry r0 = rows[ml0];
          const bool whole = m + 15 < M && (r0.pos & 15) == 0 && rows[ml0 + 15].pos == r0.pos + 15;
          const int hn = n - 2 * E.hidden, h = hn / E.head_dim, dd = hn - h * E.head_dim;
          bf16_t* vt = (bf16_t*)E.vt + ((long)h * E.head_dim + dd) * E.vt_ld;
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
      if constexpr (NCOL == 16) {
        if (E.mode == EPI_RESID) {
          // a 16-wide group under the residual update: 8 columns per lane so
          // that every lane of the wave reads, updates and writes x
          const int c8 = (lane & 1) * 8;
          const int ml = wm * WTM + i * 32 + rl;
          const int m = m0 + ml, n = nb + c8;
          if (m < M) {
            const RowEntry re = rows[ml];
            const float* g = E.mods + (long)re.req * E.mods_ld + E.gate_off + n;
            float* xo = (float*)E.out + (long)m * E.ldo + n;
            if (n + 8 <= N) {
#pragma unroll
              for (int q = 0; q < 2; ++q) {
                const float4 t = *(const float4*)&stg[rl * SP + c8 + 4 * q];
                const float4 gv = ((const float4*)g)[q];
                float4 xv = ((float4*)xo)[q];
                xv.x += gv.x * t.x;
                xv.y += gv.y * t.y;
                xv.z += gv.z * t.z;
                xv.w += gv.w * t.w;
                ((float4*)xo)[q] = xv;
              }
            } else {
#pragma unroll
              for (int q = 0; q < 8; ++q)
                if (n + q < N) xo[q] += g[q] * stg[rl * SP + c8 + q];
            }
          }
          return;
        }
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
      if (cseg < NCOL && m < M) {
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
hipError_t launch_kernel(const GemmProblem& p, int sk, hipStream_t s) {
  const long tiles = tile_count<BM, BN>(p);
  if (tiles == 0) return hipSuccess;
  GemmProblem q = p;
  q.sk_p = DTL ? sk : 1;
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, NWM, NWN, BK, STAGES, DTL>), dim3((unsigned)(tiles * q.sk_p)),
                     dim3(NWM * NWN * 64), 0, s, q);
  return hipGetLastError();
}

template <int BM, int BN, int NWM, int NWN, int BK, int STAGES>
hipError_t launch_cfg(const GemmProblem& p, int sk, hipStream_t s) {
  if (dtl_ok<BM, BN, BK>(p)) return launch_kernel<BM, BN, NWM, NWN, BK, STAGES, true>(p, sk, s);
  return launch_kernel<BM, BN, NWM, NWN, BK, STAGES, false>(p, 1, s);
}

// direct-to-LDS-only configurations (wave tiles of an odd number of 16-column
// fragments have no register path): the 256x256 register path otherwise
template <int BM, int BN, int NWM, int NWN, int BK, int STAGES>
hipError_t launch_cfg_dtl_only(const GemmProblem& p, int sk, hipStream_t s) {
  if (dtl_ok<BM, BN, BK>(p)) return launch_kernel<BM, BN, NWM, NWN, BK, STAGES, true>(p, sk, s);
  return launch_cfg<256, 256, 4, 2, 64, 2>(p, 1, s);
}

enum GemmCfg { CFG_128x64 = 0, CFG_256x256 = 1, CFG_128x128 = 2, CFG_256x128 = 3, CFG_128x256 = 4, CFG_288x192 = 5 };

// Launch-time model of the tile configurations, fitted to dit_linear timings
// on MI355X over the step's GEMM shapes (M 768 .. 16896, N 1536 .. 21504,
// K 1536 .. 15360): one CU works through ceil(tiles / 256) tiles one after
// another, a tile costing its FLOPs at a per-CU rate plus a fixed prologue /
// epilogue time.  Large tiles have the higher rate (fewer operand bytes per
// FLOP); small tiles fill the 256 CUs when the big ones would leave most idle.
struct TileModel {
  GemmCfg cfg;
  int bm, bn;
  double tflops_per_cu;
  double fixed_us;
};
// 256x128's rate is raised from its fitted 6.11 to 128x256's 6.23: inside the
// step the two tie on FLOPs per tile and 256x128 measured faster wherever the
// two competed (M 768 .. 6144, the 256 / 512 px and SD3-shaped steps 0.7 - 2.4%
// faster, the rest unchanged).
// 288x192 (12 waves of 96x48) divides 4608 x 3072 into exactly 256 tiles;
// its rate is set from the same large shapes on which 256x256 was measured
// (0.915 of 256x256's when both fill the GPU).  It is considered only for
// launches it covers in one round (see pick).
constexpr TileModel kTileModels[] = {
    {CFG_256x256, 256, 256, 7.31, 11.7},
    {CFG_256x128, 256, 128, 6.23, 8.4},
    {CFG_128x256, 128, 256, 6.23, 8.7},
    {CFG_128x128, 128, 128, 5.07, 4.1},
    {CFG_288x192, 288, 192, 6.31, 8.0},
};
// Split K: the merge adds, on the critical path, the write of a piece's
// partial sums and the last piece's read of the others' (fp32, bm x bn per
// piece) plus the arrival handshake.  A split is taken only when the model
// predicts it saves at least kSplitMinGain of the launch.
constexpr double kMergeFixedUs = 3.0;
constexpr double kMergeBytesPerUs = 40e3;
constexpr double kSplitMinGain = 0.05;
constexpr int kSplitMaxPieces = 8;

double model_us(const TileModel& t, const GemmProblem& p, int sk) {
  const long tn = (p.N + t.bn - 1) / t.bn;
  long tiles = 0;
  double work = 0.0;  // sum of piece times, microseconds
  for (int g = 0; g < p.n_groups; ++g) {
    const long tg = (long)((p.g[g].M + t.bm - 1) / t.bm) * tn;
    tiles += tg;
    work += tg * sk * (2.0 * t.bm * t.bn * p.g[g].K / sk / (t.tflops_per_cu * 1e6) + t.fixed_us);
  }
  if (tiles == 0) return 0.0;
  const long units = tiles * sk;
  double us = (double)((units + 255) / 256) * (work / units);
  if (sk > 1) us += kMergeFixedUs + (sk - 1) * 4.0 * t.bm * t.bn / kMergeBytesPerUs;
  return us;
}

bool dtl_for(GemmCfg c, const GemmProblem& p) {
  switch (c) {
    case CFG_256x256: return dtl_ok<256, 256, 64>(p);
    case CFG_256x128: return dtl_ok<256, 128, 64>(p);
    case CFG_128x256: return dtl_ok<128, 256, 64>(p);
    case CFG_128x128: return dtl_ok<128, 128, 64>(p);
    case CFG_288x192: return dtl_ok<288, 192, 64>(p);
    default: return false;
  }
}

// K may be split when the caller gave split workspace, the direct-to-LDS path
// runs, both groups share K, every piece keeps at least 4 K tiles, and the
// counters and partial-sum slots suffice.
bool split_ok(const TileModel& t, const GemmProblem& p, int sk) {
  if (p.sk_part == nullptr || p.sk_cnt == nullptr || !dtl_for(t.cfg, p)) return false;
  if (p.n_groups > 1 && p.g[0].K != p.g[1].K) return false;
  if (p.g[0].K / 64 < 4 * sk) return false;
  const long tn = (p.N + t.bn - 1) / t.bn;
  long tiles = 0;
  for (int g = 0; g < p.n_groups; ++g) tiles += (long)((p.g[g].M + t.bm - 1) / t.bm) * tn;
  return tiles <= kSplitMaxTiles && tiles * sk * t.bm * t.bn * 4L <= kSplitPartBytes;
}

struct Choice {
  GemmCfg cfg;
  int sk;
};

// pick(): the configuration and K split with the shortest modelled launch
// (its time, in microseconds, in *us when asked for; 0 for the skinny-N path,
// which the model does not cover)
Choice pick(const GemmProblem& p, double* us_out = nullptr) {
  if (us_out) *us_out = 0.0;
  if (p.N <= 64) return {CFG_128x64, 1};
  Choice best{CFG_128x128, 1};
  double best_us = 1e300;
  for (const TileModel& t : kTileModels) {
    // 288x192 has no register path, and it measured faster inside the step
    // only where its tiles fit in one round
    if (t.cfg == CFG_288x192 && (!dtl_for(t.cfg, p) || tile_count<288, 192>(p) > 256)) continue;
    const double us = model_us(t, p, 1);
    if (us < best_us) {
      best_us = us;
      best = {t.cfg, 1};
    }
  }
  Choice split = best;
  double split_us = best_us;
  for (const TileModel& t : kTileModels)
    for (int sk = 2; sk <= kSplitMaxPieces; ++sk) {
      if (t.cfg == CFG_288x192 || !split_ok(t, p, sk)) continue;  // 288x192: one-round launches only
      const double us = model_us(t, p, sk);
      if (us < split_us) {
        split_us = us;
        split = {t.cfg, sk};
      }
    }
  const bool take_split = split_us <= (1.0 - kSplitMinGain) * best_us;
  if (us_out) *us_out = take_split ? split_us : best_us;
  return take_split ? split : best;
}

// Two groups as two launches: the image group of a double block often fills
// whole rounds of 256x256 tiles by itself (4096 rows x 12288 at 1024 px,
// 16384 x 3072 at 2048 px), and the text group's few tiles then open a last
// round that is mostly idle.  Run alone, the text group takes a tiling of its
// own (smaller tiles, split K) and finishes in a fraction of a round.  The
// second launch costs one kernel boundary.
constexpr double kLaunchGapUs = 4.0;
constexpr double kGroupSplitMinGain = 0.03;

}  // namespace

bool gemm_bf16_split_groups(const GemmProblem& p) {
  if (p.n_groups < 2 || p.N <= 64) return false;
  double both = 0.0, first = 0.0, second = 0.0;
  pick(p, &both);
  GemmProblem q = p;
  q.n_groups = 1;
  pick(q, &first);
  q.g[0] = p.g[1];
  pick(q, &second);
  return first + second + kLaunchGapUs <= (1.0 - kGroupSplitMinGain) * both;
}

const char* gemm_bf16_config_name(const GemmProblem& p) {
  // "gemm_bf16_<tile>" and, for a split of K into k pieces, "..._k<k>"
  struct Names {
    std::string n[6][kSplitMaxPieces + 1];
    Names() {
      const char* base[] = {"gemm_bf16_128x64", "gemm_bf16_256x256", "gemm_bf16_128x128", "gemm_bf16_256x128",
                            "gemm_bf16_128x256", "gemm_bf16_288x192"};
      for (int c = 0; c < 6; ++c)
        for (int k = 0; k <= kSplitMaxPieces; ++k) n[c][k] = k <= 1 ? base[c] : base[c] + std::string("_k") + std::to_string(k);
    }
  };
  static const Names names;
  const Choice c = pick(p);
  return names.n[c.cfg][c.sk].c_str();
}

hipError_t launch_gemm_bf16(const GemmProblem& p, hipStream_t s) {
  const Choice c = pick(p);
  switch (c.cfg) {
    case CFG_128x64:
      return launch_cfg<128, 64, 4, 1, 64, 2>(p, 1, s);
    case CFG_256x256:
      return launch_cfg<256, 256, 4, 2, 64, 2>(p, c.sk, s);
    case CFG_256x128:
      return launch_cfg<256, 128, 4, 2, 64, 2>(p, c.sk, s);
    case CFG_128x256:
      return launch_cfg<128, 256, 2, 4, 64, 2>(p, c.sk, s);
    case CFG_288x192:
      return launch_cfg_dtl_only<288, 192, 3, 4, 64, 2>(p, c.sk, s);
    default:
      return launch_cfg<128, 128, 2, 2, 64, 2>(p, c.sk, s);
  }
}

}  // namespace dit
