// Joint text+image attention, O = softmax(Q K^T / sqrt(d)) V per head and per
// request, never materialising the L x L score matrix (online softmax over
// 64-key tiles).
//
// bf16 kernel (head_dim 128 or 64) on the gfx950 matrix cores.  Each wavefront owns
// 32 queries.  It computes the transposed score tile S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16, so every lane holds the scores of ONE query
// (column lane % 32) for half of the keys: the row max and row sum are
// register reductions plus one exchange with lane ^ 32, no LDS.  The
// probabilities are rounded to bf16 and fed straight from registers as the B
// operand of O^T = V^T P^T; for that V is kept transposed (V^T [d][keys]) and
// its 16-key groups are stored in LDS in the order the score registers hold
// them.  K and V^T tiles are double-buffered in LDS (XOR-swizzled 16-byte
// chunks); the softmax runs in the log2 domain (exp2 with log2(e)/sqrt(d)
// folded into the scale).  Blocks of one head are mapped onto one XCD so its
// K/V tiles are shared through that XCD's L2.
#include <math.h>

#include <algorithm>

#include "device_common.h"

namespace dit {

namespace {

// q-tiles of every request of the batch, longest requests first
struct AttnSched {
  int n;                     // number of requests with tokens
  int req[kMaxReq];
  int tile_off[kMaxReq + 1]; // prefix sum of q-tiles per head
};

// Lazy rescaling: the running max used for exp2 is only raised when a new
// score exceeds it by more than 2^RESCALE_SLACK; until then probabilities may
// reach 2^8, which fp32 and bf16 hold exactly as well as any other value.
// O and l always share the max they were computed with, so O / l is exact.
constexpr float RESCALE_SLACK = 8.0f;

// Scheduling pattern for a run of N (LDS read, MFMA) pairs where MFMA i uses
// read i: the first A reads, then one MFMA and one read alternately, then the
// last A MFMAs -- A fragment reads stay in flight ahead of the matrix cores.
template <int N, int A>
__device__ __forceinline__ void sched_read_ahead() {
  __builtin_amdgcn_sched_group_barrier(0x100, A, 0);
  static_for<N - A>([&](auto) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  });
  __builtin_amdgcn_sched_group_barrier(0x008, A, 0);
}

// s_waitcnt with vmcnt = 0 and the other counters left alone (gfx9 encoding).
__device__ __forceinline__ void wait_vmcnt0() { __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8)); }
// s_waitcnt with vmcnt = 0 and lgkmcnt = 0: this wave's tile loads have
// landed and its LDS fragment reads have returned
__device__ __forceinline__ void wait_vmcnt0_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(7 << 4); }

// NW waves x 32 queries per block, head dimension HD (64 or 128), BKV keys
// (64 or 128) per tile.
//
// Pipeline over key tiles j: K and V^T tiles arrive by direct-to-LDS buffer
// loads in two stages, tile j + 1 loading while tile j runs scores, softmax
// and P V in turn.
template <int NW, int HD, int STAGES, int BKV>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2)))
void attn_bf16_kernel(const AttnArgs a, const AttnSched sc) {
  static_assert(STAGES == 2, "two LDS stages, the loop is unrolled over them");
  constexpr int BQ = NW * 32;
  static_assert(HD == 64 || HD == 128, "head dim");
  static_assert(BKV == 64 || BKV == 128, "key tile");
  constexpr int CH = HD / 8;       // 16-byte chunks per key row of the K tile
  constexpr int KPI = 64 / CH;     // keys per load instruction (64 lanes x 16 bytes)
  constexpr int VCH = BKV / 8;     // 16-byte chunks per d row of the V^T tile
  constexpr int VRPI = 64 / VCH;   // V^T rows per load instruction
  constexpr int KT_U4 = BKV * CH;  // K tile: [BKV keys][CH chunks of 8 d], chunk slot swizzled by kswz
  constexpr int VT_U4 = HD * VCH;  // V^T tile: [HD d][VCH chunks of 8 key slots], chunk slot swizzled by vswz
  constexpr int KI = BKV / KPI / NW;  // K-tile load instructions per wave
  constexpr int VI = HD / VRPI / NW;  // V^T-tile load instructions per wave
  static_assert(KI * KPI * NW == BKV && VI * VRPI * NW == HD, "tile config");
  // slot of chunk c in key row `key` / V^T row `dr`: the 16 rows one
  // ds_read_b128 serves per cycle land on 16 different 16-byte bank groups
  // (an involution in c)
  auto kswz = [](int key, int c) { return HD == 128 ? c ^ (key & 15) : c ^ ((key >> 1) & 7); };
  auto vswz = [](int dr, int c) { return BKV == 128 ? c ^ (dr & 15) : c ^ ((dr >> 1) & 7); };
  __shared__ uint4 smem[STAGES][KT_U4 + VT_U4];

  const int per_head = sc.tile_off[sc.n];
  // unit (query tile x head) of this block and, on a key-split launch, its
  // key range: blocks of one XCD take consecutive indices, and a split
  // launch numbers the pieces key range first, so the blocks of one XCD
  // share K/V ranges
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  int piece = 0, id = bid;
  if (a.kv_pieces > 1) {
    piece = bid / a.units;
    id = bid - piece * a.units;
  }
  id += a.unit0;
  const int h = id / per_head;
  const int t = id - h * per_head;
  int slot = 0;
  while (slot + 1 < sc.n && t >= sc.tile_off[slot + 1]) ++slot;
  const int r = sc.req[slot];
  const int q0 = (t - sc.tile_off[slot]) * BQ;
  const int L = a.meta.joint_off[r + 1] - a.meta.joint_off[r];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hl = lane >> 5;  // lane half

  const bf16_t* __restrict__ Qg = (const bf16_t*)a.q + (long)a.qk_off[r] * a.q_tok + (long)h * a.q_head;
  const bf16_t* __restrict__ Kg = (const bf16_t*)a.k + (long)a.qk_off[r] * a.k_tok + (long)h * a.k_head;
  const bf16_t* __restrict__ Vg = (const bf16_t*)a.vt + (long)a.vt_off[r] + (long)h * a.vt_head;
  const int Lpad = a.vt_off[r + 1] - a.vt_off[r];

  // K and V^T tiles move by range-checked buffer loads straight into LDS
  // (64 lanes x 16 bytes per wave instruction, no registers).  Each lane's
  // byte offset inside a tile is fixed here; a tile only moves the buffer's
  // base.  Keys past L fall outside the K buffer of the tile and read as
  // zeros (their scores are masked); V^T columns past L lie in the request's
  // zeroed padding.
  int kvo[KI], vvo[VI];
#pragma unroll
  for (int q = 0; q < KI; ++q) {
    const int key = (wave * KI + q) * KPI + lane / CH;
    kvo[q] = (key * (int)a.k_tok + kswz(key, lane % CH) * 8) * 2;
  }
#pragma unroll
  for (int q = 0; q < VI; ++q) {
    const int dr = (wave * VI + q) * VRPI + lane / VCH;
    vvo[q] = (dr * (int)a.vt_d + vswz(dr, lane % VCH) * 8) * 2;
  }
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  char* const lbase = (char*)&smem[0][0];
  constexpr int STAGE_B = (KT_U4 + VT_U4) * 16;
  auto tile_load = [&](int j, auto stc) __attribute__((always_inline)) {
    constexpr int st = decltype(stc)::value;
    const int kv0 = j * BKV;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(Kg + (long)kv0 * a.k_tok), (short)0, ((L - 1 - kv0) * (int)a.k_tok + HD) * 2, kBufferWord3);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(Vg + kv0), (short)0, ((HD - 1) * (int)a.vt_d + Lpad - kv0) * 2, kBufferWord3);
#pragma unroll
    for (int q = 0; q < KI; ++q) {
      const int vo = kvo[q];
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rk, (__attribute__((address_space(3))) void*)(lbase + st * STAGE_B + (wv * KI + q) * KPI * CH * 16), 16,
          vo, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < VI; ++q) {
      const int vo = vvo[q];
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rv, (__attribute__((address_space(3))) void*)(lbase + st * STAGE_B + KT_U4 * 16 + (wv * VI + q) * VRPI * VCH * 16),
          16, vo, 0, 0, 0);
    }
  };

  // key tiles [jb, je) of this block (all of them unless the keys are split)
  const int nt_all = (L + BKV - 1) / BKV;
  const int jb = piece * nt_all / a.kv_pieces;
  const int je = (piece + 1) * nt_all / a.kv_pieces;
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  tile_load(jb, S0{});

  // Q fragments (B operand of S^T = K Q^T): query q0 + wave*32 + lane%32, d chunk 2*ks + lane/32
  const int qrow = q0 + wave * 32 + (lane & 31);
  bf16x8_t qf[HD / 16];
#pragma unroll
  for (int ks = 0; ks < HD / 16; ++ks) {
    uint4 u = make_uint4(0, 0, 0, 0);
    if (qrow < L) u = *(const uint4*)(Qg + (long)qrow * a.q_tok + (ks * 2 + hl) * 8);
    qf[ks] = __builtin_bit_cast(bf16x8_t, u);
  }

  f32x16_t o[HD / 32];
#pragma unroll
  for (int db = 0; db < HD / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
  float m_i = -INFINITY, l_i = 0.f;
  const float sl2 = a.scale * 1.4426950408889634f;

  // S^T of one 64-key tile: two 32x32 blocks (keys kb*32 + (i/4)*8 + hl*4 + i%4 of
  // register i, query lane % 32)
  // Per-lane LDS byte offsets of the fragment reads, fixed before the loop:
  // K fragment of k-step ks (key lane % 32 of key block 0; key block 1 is
  // 32 rows further) and V^T fragment of key step ks2 (d row lane % 32 of d
  // block 0; d block db is 32 rows further).  Stage and block offsets are
  // immediates of the reads.
  int kfo[HD / 16], vfo[BKV / 16];
#pragma unroll
  for (int ks = 0; ks < HD / 16; ++ks) kfo[ks] = ((lane & 31) * CH + kswz(lane & 31, ks * 2 + hl)) * 16;
#pragma unroll
  for (int ks2 = 0; ks2 < BKV / 16; ++ks2) {
    const int dr = lane & 31;
    vfo[ks2] = KT_U4 * 16 + (dr * VCH + vswz(dr, ks2 * 2 + hl)) * 16;
  }
  auto lds_frag = [&](int byte_off) __attribute__((always_inline)) {
    return __builtin_bit_cast(bf16x8_t, *(const uint4*)(lbase + byte_off));
  };

  // S^T of one key tile: BKV / 32 blocks of 32x32 (keys kb*32 + (i/4)*8 + hl*4 + i%4 of
  // register i, query lane % 32)
  auto scores = [&](auto stc, f32x16_t* s) __attribute__((always_inline)) {
    constexpr int st = decltype(stc)::value;
#pragma unroll
    for (int kb = 0; kb < BKV / 32; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) s[kb][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) {
#pragma unroll
      for (int kb = 0; kb < BKV / 32; ++kb) {
        // key kb*32 + lane%32 keeps the swizzle term of key lane%32 (kb*32 is a multiple of 16)
        const bf16x8_t u = lds_frag(kfo[ks] + st * STAGE_B + kb * 32 * CH * 16);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(u, qf[ks], s[kb], 0, 0, 0);
      }
    }
    // keep four fragment reads ahead of the MFMAs that consume them
    sched_read_ahead<BKV / 32 * HD / 16, 4>();
  };
  // Probabilities of one tile against the running max m_i, rounded to bf16 in
  // the order the P V operand wants them (key pairs packed by one convert);
  // returns this lane's sum of the rounded values (two bf16 products per
  // v_dot2 with (1, 1)), which is also what O accumulates.
  auto exps_pack = [&](const f32x16_t* s, bf16x8_t* pf) __attribute__((always_inline)) {
    float t0 = 0.f, t1 = 0.f;
    const bf16x2_t one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int x = 0; x < BKV / 16; ++x) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = (x & 1) * 8 + 2 * e;
        // v_exp_f32 directly: results below 2^-126 flush to zero, which the
        // softmax sum and the bf16 probabilities cannot tell from their true value
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[x >> 1][i], sl2, -m_i));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[x >> 1][i + 1], sl2, -m_i));
        const bf16x2_t pk = {(__bf16)p0, (__bf16)p1};
        if (e & 1) t1 = __builtin_amdgcn_fdot2_f32_bf16(pk, one, t1, false);
        else t0 = __builtin_amdgcn_fdot2_f32_bf16(pk, one, t0, false);
        w[e] = __builtin_bit_cast(uint32_t, pk);
      }
      pf[x] = __builtin_bit_cast(bf16x8_t, make_uint4(w[0], w[1], w[2], w[3]));
    }
    return t0 + t1;
  };
  // Online softmax of tile j's scores, then O += P V.  The probabilities are
  // first taken against the current running max; only if some lane's sum
  // exceeds 2^RESCALE_SLACK (or overflows, as on the first tile) is the true
  // row max formed, the max raised, O and l rescaled, and the tile redone.
  // O and l always share the max they were computed with, so O / l is exact.
  // Only a request's last key tile can hold keys past L, and only that tile
  // is run with masking (a run-time test inside every tile is turned by the
  // compiler into a compare and select per score on every tile).
  auto softmax_pv = [&](int j, auto stc, auto maskc, f32x16_t* s) __attribute__((always_inline)) {
    constexpr int st = decltype(stc)::value;
    if constexpr (decltype(maskc)::value) {
      const int kv0 = j * BKV;
#pragma unroll
      for (int kb = 0; kb < BKV / 32; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kv0 + kb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
          if (key >= L) s[kb][i] = -INFINITY;
        }
    }
    bf16x8_t pf[BKV / 16];
    float t = exps_pack(s, pf);
    if (__any(!(t <= (float)(1 << (int)RESCALE_SLACK)))) {
      float mx = s[0][0];
#pragma unroll
      for (int kb = 0; kb < BKV / 32; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kb][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * sl2;
      const float m_new = fmaxf(m_i, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_i - m_new);
      m_i = m_new;
      l_i *= alpha;
#pragma unroll
      for (int db = 0; db < HD / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[db][i] *= alpha;
      t = exps_pack(s, pf);
    }
    l_i += t;
#pragma unroll
    for (int ks2 = 0; ks2 < BKV / 16; ++ks2) {
#pragma unroll
      for (int db = 0; db < HD / 32; ++db) {
        // d row db*32 + lane%32 keeps the swizzle term of row lane%32
        const bf16x8_t u = lds_frag(vfo[ks2] + st * STAGE_B + db * 32 * VCH * 16);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(u, pf[ks2], o[db], 0, 0, 0);
      }
    }
    sched_read_ahead<BKV / 16 * HD / 32, 4>();
  };
  // Tile j sits in stage j % 2.  Each tile starts with the loads of tile
  // j + 1 into the other stage (freed by the barrier that ended tile j - 1)
  // and ends with this wave's loads landed and a bare barrier: after it every
  // wave's part of tile j + 1 is in LDS and no wave reads tile j any more.
  // (A __syncthreads() fence would drain nothing more but costs a wait on
  // every outstanding memory operation.)
  f32x16_t sc_t[BKV / 32];
  wait_vmcnt0();
  asm volatile("s_barrier" ::: "memory");
  // The wait before the barrier also covers the LDS reads: the compiler may
  // place the last P V MFMAs (and the waits for their V^T fragments) after the
  // barrier, and the stage those fragments come from is reloaded right after
  // it by the other waves.
  auto step = [&](int j, auto stc, auto maskc) __attribute__((always_inline)) {
    constexpr int st = decltype(stc)::value;
    if (j + 1 < je) tile_load(j + 1, std::integral_constant<int, st ^ 1>{});
    scores(stc, sc_t);
    softmax_pv(j, stc, maskc, sc_t);
    wait_vmcnt0_lgkmcnt0();
    asm volatile("s_barrier" ::: "memory");
  };
  using NoMask = std::false_type;
  using Mask = std::true_type;
  // tiles [jb, jm) hold no key past L; tile jm (if any) is the request's last
  const int jm = (je == nt_all && L % BKV != 0) ? je - 1 : je;
  int j = jb;
  for (; j + 1 < jm; j += 2) {
    step(j, S0{}, NoMask{});
    step(j + 1, S1{}, NoMask{});
  }
  if (j < jm) step(j++, S0{}, NoMask{});
  if (j < je) {
    if (((j - jb) & 1) == 0) step(j, S0{}, Mask{});
    else step(j, S1{}, Mask{});
  }

  const float l = l_i + __shfl_xor(l_i, 32, 64);
  if (a.kv_pieces > 1) {
    // one key range: O unnormalised, with its max m_i and sum l (every range
    // holds at least one key, so both are finite), for attn_merge_kernel
    const long qs = (long)bid * BQ + wave * 32 + (lane & 31);  // query slot
    float* po = a.split_buf + qs * HD;
#pragma unroll
    for (int db = 0; db < HD / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *(float4*)(po + db * 32 + g * 8 + hl * 4) =
            make_float4(o[db][g * 4 + 0], o[db][g * 4 + 1], o[db][g * 4 + 2], o[db][g * 4 + 3]);
    if (hl == 0) {
      float2* pml = (float2*)(a.split_buf + (long)a.units * a.kv_pieces * BQ * HD);
      pml[qs] = make_float2(m_i, l);
    }
    return;
  }
  if (qrow < L) {
    const float inv = 1.0f / l;
    const int row = a.o_stream_major ? padded_to_row(a.meta, r, qrow) : a.meta.joint_off[r] + qrow;
    bf16_t* og = (bf16_t*)a.o + (long)row * a.o_tok + (long)h * a.o_head;
#pragma unroll
    for (int db = 0; db < HD / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int dd = db * 32 + g * 8 + hl * 4;
        uint2 w;
        w.x = pack_bf16x2(o[db][g * 4 + 0] * inv, o[db][g * 4 + 1] * inv);
        w.y = pack_bf16x2(o[db][g * 4 + 2] * inv, o[db][g * 4 + 3] * inv);
        *(uint2*)(og + dd) = w;
      }
  }
}

// Merge of a key-split launch: for each query of unit unit0 + blockIdx.x, the
// KP key ranges' unnormalised outputs O_p with maxima m_p (log2 domain) and
// sums l_p combine as O = sum_p 2^(m_p - M) O_p / sum_p 2^(m_p - M) l_p with
// M = max_p m_p, added in piece order.  Two threads per query, HD / 2
// dimensions each.
template <int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(const AttnArgs a, const AttnSched sc) {
  constexpr int BQ = 128;
  constexpr int DH = HD / 2;
  const int u = blockIdx.x;
  const int id = a.unit0 + u;
  const int per_head = sc.tile_off[sc.n];
  const int h = id / per_head;
  const int t = id - h * per_head;
  int slot = 0;
  while (slot + 1 < sc.n && t >= sc.tile_off[slot + 1]) ++slot;
  const int r = sc.req[slot];
  const int ql = threadIdx.x >> 1, part = threadIdx.x & 1;
  const int qrow = (t - sc.tile_off[slot]) * BQ + ql;
  const int L = a.meta.joint_off[r + 1] - a.meta.joint_off[r];
  if (qrow >= L) return;
  const int KP = a.kv_pieces, U = a.units;
  const float2* pml = (const float2*)(a.split_buf + (long)U * KP * BQ * HD);
  float M = -INFINITY;
  for (int p = 0; p < KP; ++p) M = fmaxf(M, pml[(long)(p * U + u) * BQ + ql].x);
  float acc[DH];
#pragma unroll
  for (int i = 0; i < DH; ++i) acc[i] = 0.f;
  float lsum = 0.f;
  for (int p = 0; p < KP; ++p) {
    const long qs = (long)(p * U + u) * BQ + ql;
    const float2 ml = pml[qs];
    const float w = exp2f(ml.x - M);
    lsum = fmaf(w, ml.y, lsum);
    const float4* src = (const float4*)(a.split_buf + qs * HD + part * DH);
#pragma unroll
    for (int c = 0; c < DH / 4; ++c) {
      const float4 v = src[c];
      acc[4 * c + 0] = fmaf(w, v.x, acc[4 * c + 0]);
      acc[4 * c + 1] = fmaf(w, v.y, acc[4 * c + 1]);
      acc[4 * c + 2] = fmaf(w, v.z, acc[4 * c + 2]);
      acc[4 * c + 3] = fmaf(w, v.w, acc[4 * c + 3]);
    }
  }
  const float inv = 1.0f / lsum;
  const int row = a.o_stream_major ? padded_to_row(a.meta, r, qrow) : a.meta.joint_off[r] + qrow;
  bf16_t* og = (bf16_t*)a.o + (long)row * a.o_tok + (long)h * a.o_head + part * DH;
#pragma unroll
  for (int c = 0; c < DH / 8; ++c) {
    uint4 w;
    w.x = pack_bf16x2(acc[8 * c + 0] * inv, acc[8 * c + 1] * inv);
    w.y = pack_bf16x2(acc[8 * c + 2] * inv, acc[8 * c + 3] * inv);
    w.z = pack_bf16x2(acc[8 * c + 4] * inv, acc[8 * c + 5] * inv);
    w.w = pack_bf16x2(acc[8 * c + 6] * inv, acc[8 * c + 7] * inv);
    *(uint4*)(og + 8 * c) = w;
  }
}

// ----------------------------------------------------------------------------
// fp32 attention (head_dim 64) for fp32 models: 64 queries per block, four
// lanes per query (lane part p holds dims 16p .. 16p + 15 of q and O), K and V
// tiles of 64 keys in LDS (rows of 16 float4, padded to 17 so the tile stores
// of a wave spread over the banks), and the online softmax taken per tile in
// fp32: all 64 scores of a tile (partial dot products summed over the quad),
// one rescale of O and l, then O += P V.  exp2 of a log2(e)-scaled argument
// adds one rounding of the argument (about 2e-6 relative at the scores met).
constexpr int FD = 64;
constexpr int FQ = 64;

__global__ __launch_bounds__(256) void attn_f32_kernel(const AttnArgs a, const AttnSched sc) {
  constexpr int F4 = FD / 4;  // float4 per row
  constexpr float kLog2e = 1.4426950408889634f;
  __shared__ float4 Ksh[64][F4 + 1];
  __shared__ float4 Vsh[64][F4 + 1];
  const int per_head = sc.tile_off[sc.n];
  const int h = blockIdx.x / per_head;
  const int t = blockIdx.x - h * per_head;
  int slot = 0;
  while (slot + 1 < sc.n && t >= sc.tile_off[slot + 1]) ++slot;
  const int r = sc.req[slot];
  const int q0 = (t - sc.tile_off[slot]) * FQ;
  const int L = a.meta.joint_off[r + 1] - a.meta.joint_off[r];
  const int tid = threadIdx.x;
  const int part = tid & 3;  // the quad of a query is four consecutive lanes of one wave
  const int qrow = q0 + (tid >> 2);

  const float* Qg = (const float*)a.q + (long)a.qk_off[r] * a.q_tok + (long)h * a.q_head;
  const float* Kg = (const float*)a.k + (long)a.qk_off[r] * a.k_tok + (long)h * a.k_head;
  const float* Vg = (const float*)a.vt + (long)a.vt_off[r] + (long)h * a.vt_head;

  float4 q[4], o[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    q[c] = (qrow < L) ? *(const float4*)(Qg + (long)qrow * a.q_tok + 16 * part + 4 * c)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
    o[c] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  const float sl2 = a.scale * kLog2e;
  float m = -INFINITY, l = 0.f;  // m in the log2 domain
  for (int kv0 = 0; kv0 < L; kv0 += 64) {
    __syncthreads();
    // Each operand's tile arrives as 4 float4 loads per thread, all in flight
    // before the LDS stores.  K rows past L re-read row L - 1 (their scores are
    // masked); V^T is read in slot order, 64 slots of the request's padded
    // columns per d, and slot s holds key vt_slot(s) (an involution).
    {
      float4 tq[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = tid + u * 256;
        tq[u] = *(const float4*)(Kg + (long)min(kv0 + (idx >> 4), L - 1) * a.k_tok + (idx & 15) * 4);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = tid + u * 256;
        Ksh[idx >> 4][idx & 15] = tq[u];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = tid + u * 256;
        tq[u] = *(const float4*)(Vg + (long)(idx >> 4) * a.vt_d + kv0 + (idx & 15) * 4);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = tid + u * 256, c = idx >> 4, s0 = kv0 + (idx & 15) * 4;
        ((float*)Vsh[vt_slot(s0) - kv0])[c] = tq[u].x;
        ((float*)Vsh[vt_slot(s0 + 1) - kv0])[c] = tq[u].y;
        ((float*)Vsh[vt_slot(s0 + 2) - kv0])[c] = tq[u].z;
        ((float*)Vsh[vt_slot(s0 + 3) - kv0])[c] = tq[u].w;
      }
    }
    __syncthreads();
    const int nk = min(64, L - kv0);
    float s[64];
    float mx = m;
#pragma unroll
    for (int j = 0; j < 64; ++j) {
      float d = 0.f;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float4 k4 = Ksh[j][4 * part + c];
        d = fmaf(q[c].x, k4.x, fmaf(q[c].y, k4.y, fmaf(q[c].z, k4.z, fmaf(q[c].w, k4.w, d))));
      }
      d += __shfl_xor(d, 1, 64);
      d += __shfl_xor(d, 2, 64);
      s[j] = j < nk ? d * sl2 : -INFINITY;
      mx = fmaxf(mx, s[j]);
    }
    // mx is finite: the tile holds at least one key
    const float al = exp2f(m - mx);
    float ps = 0.f;
#pragma unroll
    for (int j = 0; j < 64; ++j) {
      s[j] = exp2f(s[j] - mx);
      ps += s[j];
    }
    l = l * al + ps;
    m = mx;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float4 acc = make_float4(o[c].x * al, o[c].y * al, o[c].z * al, o[c].w * al);
#pragma unroll
      for (int j = 0; j < 64; ++j) {
        const float4 v = Vsh[j][4 * part + c];
        acc.x = fmaf(s[j], v.x, acc.x);
        acc.y = fmaf(s[j], v.y, acc.y);
        acc.z = fmaf(s[j], v.z, acc.z);
        acc.w = fmaf(s[j], v.w, acc.w);
      }
      o[c] = acc;
    }
  }
  if (qrow < L) {
    const int row = a.o_stream_major ? padded_to_row(a.meta, r, qrow) : a.meta.joint_off[r] + qrow;
    float* og = (float*)a.o + (long)row * a.o_tok + (long)h * a.o_head + 16 * part;
    const float inv = 1.0f / l;
#pragma unroll
    for (int c = 0; c < 4; ++c)
      *(float4*)(og + 4 * c) = make_float4(o[c].x * inv, o[c].y * inv, o[c].z * inv, o[c].w * inv);
  }
}

AttnSched make_sched(const BatchMeta& m, int bq) {
  AttnSched sc{};
  int order[kMaxReq];
  int n = 0;
  for (int r = 0; r < m.n_req; ++r)
    if (m.joint_off[r + 1] > m.joint_off[r]) order[n++] = r;
  // longest requests first: their tiles take longest, start them early
  for (int i = 1; i < n; ++i)
    for (int j = i; j > 0; --j) {
      const int a = order[j - 1], b = order[j];
      if (m.joint_off[b + 1] - m.joint_off[b] > m.joint_off[a + 1] - m.joint_off[a]) {
        order[j - 1] = b;
        order[j] = a;
      }
    }
  sc.n = n;
  sc.tile_off[0] = 0;
  for (int i = 0; i < n; ++i) {
    const int r = order[i];
    sc.req[i] = r;
    const int L = m.joint_off[r + 1] - m.joint_off[r];
    sc.tile_off[i + 1] = sc.tile_off[i] + (L + bq - 1) / bq;
  }
  return sc;
}

}  // namespace

// keys per tile of the bf16 kernel; a request's V^T columns are padded to a
// multiple of kSeqPad, so a tile never reads past them
constexpr int kKeyTile = 64;
static_assert(kSeqPad % kKeyTile == 0, "V^T padding");

template <int NW, int HD>
hipError_t launch_attn_cfg(const AttnArgs& a, hipStream_t s) {
  const AttnSched sc = make_sched(a.meta, NW * 32);
  const long blocks = (long)sc.tile_off[sc.n] * a.heads;
  if (blocks == 0) return hipSuccess;
  AttnArgs b = a;
  b.unit0 = 0;
  b.units = (int)blocks;
  b.kv_pieces = 1;
  hipLaunchKernelGGL((attn_bf16_kernel<NW, HD, 2, kKeyTile>), dim3((unsigned)blocks), dim3(NW * 64), 0, s, b, sc);
  return hipGetLastError();
}

// Key split of the last round.  A launch of U 128-query units on the 512
// block slots of the GPU (two per CU) runs floor(U / 512) full rounds and a
// last one of T = U mod 512 units.  A unit alone on its CU runs about twice
// as fast as one of a pair, so a last round of up to 256 units costs about
// what its share of work would; below a quarter round, though, it still
// costs more (measured on MI355X at 16 384 tokens and head dim 128: 0.25 of
// a round of units took 0.37 of a round's time, 0.5 took 0.5).  When
// T <= 128 after R >= 2 full rounds, those T units instead run as T x P
// blocks of one key range each (P = floor(512 / T) >= 4 pieces, 1/P as long),
// and a merge kernel combines the pieces.  Measured against the unsplit
// launch at 16 384-17 152 tokens and 24-25 heads: 1.1-1.7% faster for
// T = 24-128 (P = 21-4), equal at P = 3 and 1% slower at P = 2, hence the
// bound.  Requests of one length only (the units of a mixed batch differ in
// cost), head dim 128.
struct SplitPlan {
  int main_units, tail_units, pieces;  // pieces 0: no split
};

constexpr int kAttnSlots = 2 * 256;  // 128-query blocks resident per GPU (two per CU, 256 CUs)

SplitPlan split_plan(const BatchMeta& m, int heads, int head_dim) {
  SplitPlan p{0, 0, 0};
  if (head_dim != 128) return p;
  const AttnSched sc = make_sched(m, 128);
  if (sc.n == 0) return p;
  const int L0 = m.joint_off[sc.req[0] + 1] - m.joint_off[sc.req[0]];
  for (int i = 1; i < sc.n; ++i)
    if (m.joint_off[sc.req[i] + 1] - m.joint_off[sc.req[i]] != L0) return p;
  const long units = (long)sc.tile_off[sc.n] * heads;
  const long full = units / kAttnSlots, tail = units % kAttnSlots;
  if (full < 2 || tail == 0 || 4 * tail > kAttnSlots) return p;
  const int key_tiles = (L0 + kKeyTile - 1) / kKeyTile;
  const int pieces = (int)std::min<long>(kAttnSlots / tail, key_tiles);
  if (pieces < 2) return p;
  p.main_units = (int)(full * kAttnSlots);
  p.tail_units = (int)tail;
  p.pieces = pieces;
  return p;
}

size_t split_bytes(const SplitPlan& p, int head_dim) {
  return p.pieces ? (size_t)p.tail_units * p.pieces * 128 * (head_dim + 2) * sizeof(float) : 0;
}

// Measured on MI355X: software pipelines that overlap a tile's softmax with
// the next tile's score MFMAs (255 VGPRs, spills) or with the previous tile's
// P V MFMAs (separate K and V^T rings of 2 or 4 stages, ~205 VGPRs) gave the
// same bits and were no faster where attention matters most (16 896 tokens),
// so the plain order with 2 buffers is used.
// Block shape at head dim 128.  Blocks of 128 queries (4 waves) run two per
// CU; their last round of a launch holds the leftover blocks, and when these
// are at most one per CU each runs alone on its CU, much faster than as one
// of two.  Blocks of 256 queries (8 waves, one per CU) read each K/V tile once
// for twice the queries but get no such lone tail.  So with U units (128
// queries x heads) on 2 x 256 block slots, the 128-query blocks win when the
// 256-query launch's last round (of 256 slots) is at most half full and the
// 256-query blocks otherwise: with an even number of 128-query tiles per
// request that is frac(U / 512) <= 1/2; with an odd number each request
// adds a half-empty 256-query block (at 19 072 tokens, 24 heads: 1800
// blocks, a last round of 8; the 128-query blocks are 6% faster there).
// Measured on MI355X (in-process A/B) at
// 16 896 tokens: 6 heads (U = 792) 256-query blocks -11%, 12 heads (1584)
// +4%, 18 heads
// (2376) -7%, 24 heads (3168) +2%; at 4608 tokens: 24 heads (864) -4%,
// 48 heads (1728) +3%; whole steps at 256 px (144) +1.8% and 512 px (288)
// -0.9%.  The rule assumes equal units, i.e. requests of one length; for a
// batch of mixed lengths (longest first, so the last round holds the short
// units) the 128-query blocks are kept (the packed 256-2048 px step: +0.6%
// with 256-query blocks).  At head dim 64 (half the registers, so two
// 256-query blocks fit on a CU) the 256-query blocks stay ahead until the
// launch has 2048 units.
template <int HD>
hipError_t launch_attn_hd(const AttnArgs& a, hipStream_t s) {
  const SplitPlan sp = a.split_buf ? split_plan(a.meta, a.heads, HD) : SplitPlan{0, 0, 0};
  if (sp.pieces) {
    const AttnSched sc = make_sched(a.meta, 128);
    AttnArgs b = a;
    b.unit0 = 0;
    b.units = sp.main_units;
    b.kv_pieces = 1;
    hipLaunchKernelGGL((attn_bf16_kernel<4, HD, 2, kKeyTile>), dim3((unsigned)sp.main_units), dim3(256), 0, s, b, sc);
    b.unit0 = sp.main_units;
    b.units = sp.tail_units;
    b.kv_pieces = sp.pieces;
    hipLaunchKernelGGL((attn_bf16_kernel<4, HD, 2, kKeyTile>), dim3((unsigned)(sp.tail_units * sp.pieces)), dim3(256), 0, s, b,
                       sc);
    hipLaunchKernelGGL((attn_merge_kernel<HD>), dim3((unsigned)sp.tail_units), dim3(256), 0, s, b, sc);
    return hipGetLastError();
  }
  const AttnSched sc4 = make_sched(a.meta, 4 * 32);
  const long units = (long)sc4.tile_off[sc4.n] * a.heads;
  bool wide;
  if (HD == 128) {
    bool equal = true;
    const int L0 = a.meta.joint_off[sc4.req[0] + 1] - a.meta.joint_off[sc4.req[0]];
    for (int i = 1; i < sc4.n; ++i)
      equal = equal && a.meta.joint_off[sc4.req[i] + 1] - a.meta.joint_off[sc4.req[i]] == L0;
    // fill of the 256-query launch's own last round (its block count is not
    // units / 2 when a request has an odd number of 128-query tiles)
    const AttnSched sc8 = make_sched(a.meta, 8 * 32);
    const long units8 = (long)sc8.tile_off[sc8.n] * a.heads;
    constexpr long kSlots8 = 256;  // 256-query blocks resident per GPU (one per CU)
    wide = equal && 2 * (units8 % kSlots8) > kSlots8;
  } else {
    wide = units < 2048;
  }
  if (wide) return launch_attn_cfg<8, HD>(a, s);
  return launch_attn_cfg<4, HD>(a, s);
}

hipError_t launch_attention_bf16(const AttnArgs& a, hipStream_t s) {
  if (a.head_dim == 128) return launch_attn_hd<128>(a, s);
  if (a.head_dim == 64) return launch_attn_hd<64>(a, s);
  return hipErrorInvalidValue;
}

size_t attn_split_bytes(const BatchMeta& m, int heads, int head_dim) {
  return split_bytes(split_plan(m, heads, head_dim), head_dim);
}

hipError_t launch_attention_f32(const AttnArgs& a, hipStream_t s) {
  if (a.head_dim != FD) return hipErrorInvalidValue;
  const AttnSched sc = make_sched(a.meta, FQ);
  const long blocks = (long)sc.tile_off[sc.n] * a.heads;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(attn_f32_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a, sc);
  return hipGetLastError();
}

}  // namespace dit
