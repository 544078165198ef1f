// Entropy coding of the quantised latent (Fig. 4 "AE" / "AD", Fig. 6): rANS
// (Duda 2013, range variant: 32-bit state in [2^16, 2^32), 16-bit words,
// M = 2^16) on quantised-scale Gaussian tables.
//
// A stream is 8192 symbols coded by the 64 lanes of one wave in lock step:
// symbol i of the stream belongs to lane i % 64 at step i / 64, so symbol and
// scale-index loads are coalesced.  At every (step, sub-symbol) the lanes that
// move a word do so in lane order (ballot + popcount give each its slot), so a
// stream is one contiguous run of words.  Escaped symbols (|q| beyond the
// table) continue with uniform sub-symbols: the sign, the digit count, then
// the hex digits of |q| - R - 1, most significant first.
//
// k_rans_encode  one wave per stream: encodes backwards into the stream's
//                scratch slot, words ending at the slot's end
// k_rans_frame   one workgroup: prefix sum of the stream lengths, container
//                header and length table
// k_rans_pack    one workgroup per stream: copies the words into the container
// k_rans_index   one workgroup: checks a container, prefix sum of its lengths
// k_rans_decode  one wave per stream: decodes forward, every word read bounded
//                by the stream's length; flags a truncated or inconsistent
//                stream instead of reading past it
#include "common.hpp"
#include "internal.hpp"

namespace nc {

namespace {

constexpr uint32_t kRansL = 1u << 16;

struct Sub {
  uint32_t c, f;
};

// Sub-symbol u of a symbol (decoding order): u = 0 the table entry (or ESC),
// then for an escape the sign (M / 2 each), the digit count minus one
// (M / 4 each) and the digits (M / 16 each).
__device__ __forceinline__ Sub rans_sub(int u, uint32_t ent, bool neg, int nd, uint32_t v) {
  if (u == 0) return {ent >> 16, ent & 0xFFFFu};
  if (u == 1) return {neg ? 32768u : 0u, 32768u};
  if (u == 2) return {(uint32_t)(nd - 1) * 16384u, 16384u};
  return {((v >> (4 * (nd - 1 - (u - 3)))) & 15u) * 4096u, 4096u};
}

__device__ __forceinline__ int wave_max(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = max(v, __shfl_xor(v, off, 64));
  return v;
}

}  // namespace

__global__ __launch_bounds__(256) void k_rans_encode(const int16_t* q, const uint8_t* kidx, int64_t n, RansTab t,
                                                   uint16_t* scratch, int64_t max_words, uint32_t* lens) {
  const int lane = threadIdx.x & 63;
  const int64_t s = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t ns = (n + kRansStream - 1) / kRansStream;
  if (s >= ns) return;  // whole waves
  const int64_t base = s * kRansStream;
  const int cnt = (int)min((int64_t)kRansStream, n - base);
  const int steps = (cnt + 63) / 64;
  uint16_t* end = scratch + (s + 1) * max_words;
  int64_t p = 0;  // words written, counted back from the end
  uint32_t x = kRansL;
  for (int st = steps - 1; st >= 0; --st) {
    const int li = st * 64 + lane;
    const bool act = li < cnt;
    int nsub = 0, nd = 1;
    uint32_t ent = 0, v = 0;
    bool neg = false;
    if (act) {
      const int qv = q[base + li];
      const int k = min((int)kidx[base + li], kCoderScales - 1);
      const int R = t.R[k];
      const int off = t.off[k];
      if (qv >= -R && qv <= R) {
        ent = t.ent[off + qv + R];
        nsub = 1;
      } else {
        ent = t.ent[off + 2 * R + 1];
        neg = qv < 0;
        v = (uint32_t)(abs(qv) - R - 1);
        while (nd < 4 && v >= (1u << (4 * nd))) ++nd;
        nsub = 3 + nd;
      }
    }
    const int maxsub = wave_max(nsub);
    for (int u = maxsub - 1; u >= 0; --u) {
      const bool part = u < nsub;
      const Sub sb = rans_sub(u, ent, neg, nd, v);
      const bool emit = part && x >= (sb.f << 16);
      const uint64_t m = __ballot(emit);
      const int cw = __popcll(m);
      if (emit) {
        const int rank = __popcll(m & ((1ull << lane) - 1));
        end[-(p + cw) + rank] = (uint16_t)(x & 0xFFFFu);
        x >>= 16;
      }
      p += cw;
      if (part) x = (x / sb.f) * 65536u + (x % sb.f) + sb.c;
    }
  }
  // the 64 final states open the stream: lane l at words 2l (high) and 2l + 1
  end[-(p + 128) + 2 * lane] = (uint16_t)(x >> 16);
  end[-(p + 128) + 2 * lane + 1] = (uint16_t)(x & 0xFFFFu);
  p += 128;
  if (lane == 0) lens[s] = (uint32_t)p;
}

// Block-wide exclusive prefix sum of one value per thread (1024 threads).
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* total, uint32_t* sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_up(inc, off, 64);
    if (lane >= off) inc += o;
  }
  if (lane == 63) sh[wave] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t acc = 0;
    for (int w = 0; w < 16; ++w) {
      const uint32_t t = sh[w];
      sh[w] = acc;
      acc += t;
    }
    sh[16] = acc;
  }
  __syncthreads();
  const uint32_t r = sh[wave] + inc - v;
  *total = sh[16];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(1024) void k_rans_frame(const uint32_t* lens, int64_t n, uint32_t* offs, uint8_t* out,
                                                   uint64_t* nbytes) {
  __shared__ uint32_t sh[17];
  const int ns = (int)((n + kRansStream - 1) / kRansStream);
  uint16_t* ltab = (uint16_t*)(out + kRansHeader);
  uint32_t carry = 0;
  for (int b = 0; b < ns; b += 1024) {
    const int i = b + threadIdx.x;
    const uint32_t v = i < ns ? lens[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_excl_scan(v, &tot, sh);
    if (i < ns) {
      offs[i] = carry + ex;
      ltab[i] = (uint16_t)v;
    }
    carry += tot;
  }
  if (threadIdx.x == 0) {
    uint32_t* h = (uint32_t*)out;
    h[0] = kRansMagic;
    h[1] = kRansVersion;
    h[2] = (uint32_t)n;
    h[3] = (uint32_t)kRansStream;
    h[4] = (uint32_t)ns;
    if (ns & 1) ltab[ns] = 0;  // pad to 4 bytes
    *nbytes = (uint64_t)rans_payload_offset(ns) + 2ull * carry;
  }
}

__global__ __launch_bounds__(256) void k_rans_pack(const uint16_t* scratch, int64_t max_words, const uint32_t* lens,
                                                 const uint32_t* offs, int64_t n, uint8_t* out) {
  const int ns = (int)((n + kRansStream - 1) / kRansStream);
  const int s = blockIdx.x;
  if (s >= ns) return;
  const uint32_t len = lens[s];
  const uint16_t* src = scratch + (int64_t)(s + 1) * max_words - len;
  uint16_t* dst = (uint16_t*)(out + rans_payload_offset(ns)) + offs[s];
  for (uint32_t i = threadIdx.x; i < len; i += 256) dst[i] = src[i];
}

__global__ __launch_bounds__(1024) void k_rans_index(const uint8_t* in, uint64_t in_bytes, int64_t n, uint32_t* offs,
                                                   uint32_t* lens, int32_t* status) {
  __shared__ uint32_t sh[17];
  __shared__ int bad;
  const int ns = (int)((n + kRansStream - 1) / kRansStream);
  if (threadIdx.x == 0) {
    bad = 0;
    if (in_bytes < (uint64_t)rans_payload_offset(ns)) {
      bad = 1;
    } else {
      const uint32_t* h = (const uint32_t*)in;
      bad = !(h[0] == kRansMagic && h[1] == kRansVersion && h[2] == (uint32_t)n && h[3] == (uint32_t)kRansStream &&
              h[4] == (uint32_t)ns);
    }
  }
  __syncthreads();
  const bool ok = !bad;
  const uint16_t* ltab = (const uint16_t*)(in + kRansHeader);
  uint32_t carry = 0;
  for (int b = 0; b < ns; b += 1024) {
    const int i = b + threadIdx.x;
    const uint32_t v = (ok && i < ns) ? ltab[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_excl_scan(v, &tot, sh);
    if (i < ns) {
      offs[i] = carry + ex;
      lens[i] = v;
    }
    carry += tot;
  }
  if (threadIdx.x == 0) {
    int st = bad ? 1 : 0;
    if (!bad && (uint64_t)rans_payload_offset(ns) + 2ull * carry > in_bytes) st = 1;
    status[0] = st;
    status[1] = 0;
  }
}

__global__ __launch_bounds__(256) void k_rans_decode(const uint8_t* in, const uint8_t* kidx, int64_t n, RansTab t,
                                                   const uint32_t* offs, const uint32_t* lens, int16_t* q,
                                                   int32_t* status) {
  const int lane = threadIdx.x & 63;
  const int64_t s = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t ns = (n + kRansStream - 1) / kRansStream;
  if (s >= ns) return;
  const int64_t base = s * kRansStream;
  const int cnt = (int)min((int64_t)kRansStream, n - base);
  const int steps = (cnt + 63) / 64;
  const bool head_ok = status[0] == 0;  // status[0]: container check, status[1]: stream errors
  const uint32_t len = head_ok ? lens[s] : 0u;
  const uint16_t* w = (const uint16_t*)(in + rans_payload_offset((int)ns)) + (head_ok ? offs[s] : 0u);
  int err = 0;
  auto word = [&](uint32_t i) -> uint32_t {
    if (i < len) return w[i];
    err |= 2;
    return 0u;
  };
  uint32_t x = (word(2 * lane) << 16) | word(2 * lane + 1);
  uint32_t pos = 128;
  // one decoding step of a sub-symbol with start c and frequency f, plus the
  // lane-ordered renormalisation reads
  auto advance = [&](bool part, uint32_t c, uint32_t f) {
    if (part) x = f * (x >> 16) + (x & 0xFFFFu) - c;
    const bool need = part && x < kRansL;
    const uint64_t m = __ballot(need);
    if (need) x = (x << 16) | word(pos + __popcll(m & ((1ull << lane) - 1)));
    pos += __popcll(m);
  };
  for (int st = 0; st < steps; ++st) {
    const int li = st * 64 + lane;
    const bool act = li < cnt;
    int k = 0, R = 0, off = 0, qv = 0;
    bool esc = false;
    uint32_t c = 0, f = 1;
    if (act) {
      k = min((int)kidx[base + li], kCoderScales - 1);
      R = t.R[k];
      off = t.off[k];
      // entry holding the slot: the bucket bounds it, a binary search finds it
      const uint32_t slot = x & 0xFFFFu;
      const int b = (int)(slot >> 8);
      int lo = t.bkt[k * 257 + b], hi = t.bkt[k * 257 + b + 1];
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((t.ent[off + mid] >> 16) <= slot) lo = mid;
        else hi = mid - 1;
      }
      const uint32_t e = t.ent[off + lo];
      c = e >> 16;
      f = e & 0xFFFFu;
      esc = lo == 2 * R + 1;
      qv = lo - R;
    }
    advance(act, c, f);
    if (__ballot(esc)) {
      bool neg = false;
      int nd = 0;
      uint32_t v = 0;
      // sign, digit count
      {
        const uint32_t u = esc ? (x & 0xFFFFu) >> 15 : 0u;
        advance(esc, u * 32768u, 32768u);
        neg = u != 0;
      }
      {
        const uint32_t u = esc ? (x & 0xFFFFu) >> 14 : 0u;
        advance(esc, u * 16384u, 16384u);
        nd = (int)u + 1;
      }
      const int maxd = wave_max(esc ? nd : 0);
      for (int d = 0; d < maxd; ++d) {
        const bool part = esc && d < nd;
        const uint32_t u = part ? (x & 0xFFFFu) >> 12 : 0u;
        advance(part, u * 4096u, 4096u);
        if (part) v = v * 16u + u;
      }
      if (esc) {
        const int mag = R + 1 + (int)v;
        qv = neg ? -mag : mag;
      }
    }
    if (act) q[base + li] = (int16_t)max(min(qv, 32767), -32768);
  }
  if (head_ok && (x != kRansL || pos != len)) err |= 4;
  if (err) atomicOr(status + 1, err);
}

__global__ void k_rans_status(const int32_t* status, int32_t* out) { *out = status[0] | status[1]; }

hipError_t launch_rans_encode(const int16_t* q, const uint8_t* k, int64_t n, const RansTab& t, uint16_t* scratch,
                              int64_t max_words, uint32_t* lens, uint32_t* offs, uint8_t* out, uint64_t* nbytes,
                              hipStream_t st) {
  const int64_t ns = (n + kRansStream - 1) / kRansStream;
  if (ns <= 0 || ns > 65535) return hipErrorInvalidValue;
  launch(k_rans_encode, dim3((unsigned)((ns + 3) / 4)), dim3(256), st, q, k, n, t, scratch, max_words, lens);
  launch(k_rans_frame, dim3(1), dim3(1024), st, (const uint32_t*)lens, n, offs, out, nbytes);
  launch(k_rans_pack, dim3((unsigned)ns), dim3(256), st, (const uint16_t*)scratch, max_words, (const uint32_t*)lens,
         (const uint32_t*)offs, n, out);
  return hipGetLastError();
}

hipError_t launch_rans_decode(const uint8_t* in, uint64_t in_bytes, const uint8_t* k, int64_t n, const RansTab& t,
                              uint32_t* offs, uint32_t* lens, int16_t* q, int32_t* status, int32_t* status_out,
                              hipStream_t st) {
  const int64_t ns = (n + kRansStream - 1) / kRansStream;
  if (ns <= 0 || ns > 65535) return hipErrorInvalidValue;
  launch(k_rans_index, dim3(1), dim3(1024), st, in, in_bytes, n, offs, lens, status);
  launch(k_rans_decode, dim3((unsigned)((ns + 3) / 4)), dim3(256), st, in, k, n, t, (const uint32_t*)offs,
         (const uint32_t*)lens, q, status);
  if (status_out) launch(k_rans_status, dim3(1), dim3(1), st, (const int32_t*)status, status_out);
  return hipGetLastError();
}

}  // namespace nc
