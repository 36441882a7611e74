// exp64.hip -- Exp-MCN over binary64 components with a correctly rounded binary64
// component exponential, on gfx950.
//
// The component exponential (the paper's algorithm calls the framework's exp; the
// reading used here is the correctly rounded one, the only choice that makes the
// result a function of the inputs alone) follows Tang's table method:
//   x = (64 k + j) ln2/64 + r, j in [0, 64), |r| <= ln2/128 + tiny,
//   e^x = 2^k 2^(j/64) e^r.
// First stage, double-double: r from a three-part ln2/64 (the first part has 36
// significant bits, so its product with |N| < 2^17 is exact), e^r = 1 + r + r^2/2 +
// r^3 q(r) with r + r^2/2 kept exact as a double-double and q(r) = 1/3! + ... + r^6/9!
// in binary64 Horner form (the terms beyond degree 9 are below 2^-96), the table value
// 2^(j/64) as a double-double read from a copy in LDS.  Its relative error is below
// 2^-75; the result is final when every value within 2^-69 (relative) of it rounds to
// the same binary64 number (to the same multiple of 2^-1074 for results below 2^-1021).
// When every argument of a wavefront is below 2^-27 in magnitude (the low components of
// an expansion), a shorter first stage, 1 + x + x^2/2 + x^3/6, takes the same test.
// Otherwise -- about one argument in 2^16 -- the second stage evaluates e^x in 192-bit
// fixed point (176 fraction bits: ln2/64 and 2^(j/64) to 176 bits, Taylor series of e^r
// to degree 20, relative error below 2^-165) and rounds those bits to nearest.  e^x is
// transcendental for every non-zero binary64 x, so it never lies on a rounding boundary,
// and no binary64 argument brings it within 2^-165 of one.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "exp32.hpp"
#include "mcf_arith.hpp"
#include "mcf_internal.hpp"

namespace mcf {
namespace {

// ln2/64 = L1 + L2 + L3 (L1: 36 significant bits) and 64/ln2, binary64.
constexpr double EXP64_L1 = 0x1.62e42fefa0000p-7;
constexpr double EXP64_L2 = 0x1.cf79abc9e3b3ap-46;
constexpr double EXP64_L3 = -0x1.ff0342542fc33p-100;
constexpr double EXP64_INV = 0x1.71547652b82fep+6;

// 2^(j/64) = hi + lo, binary64 pairs, j = 0 .. 63.
__constant__ double EXP64_T_DD[64][2] = {
    {0x1.0000000000000p+0, 0x0.0p+0},
    {0x1.02c9a3e778061p+0, -0x1.19083535b085dp-56},
    {0x1.059b0d3158574p+0, 0x1.d73e2a475b465p-55},
    {0x1.0874518759bc8p+0, 0x1.186be4bb284ffp-57},
    {0x1.0b5586cf9890fp+0, 0x1.8a62e4adc610bp-54},
    {0x1.0e3ec32d3d1a2p+0, 0x1.03a1727c57b53p-59},
    {0x1.11301d0125b51p+0, -0x1.6c51039449b3ap-54},
    {0x1.1429aaea92de0p+0, -0x1.32fbf9af1369ep-54},
    {0x1.172b83c7d517bp+0, -0x1.19041b9d78a76p-55},
    {0x1.1a35beb6fcb75p+0, 0x1.e5b4c7b4968e4p-55},
    {0x1.1d4873168b9aap+0, 0x1.e016e00a2643cp-54},
    {0x1.2063b88628cd6p+0, 0x1.dc775814a8495p-55},
    {0x1.2387a6e756238p+0, 0x1.9b07eb6c70573p-54},
    {0x1.26b4565e27cddp+0, 0x1.2bd339940e9d9p-55},
    {0x1.29e9df51fdee1p+0, 0x1.612e8afad1255p-55},
    {0x1.2d285a6e4030bp+0, 0x1.0024754db41d5p-54},
    {0x1.306fe0a31b715p+0, 0x1.6f46ad23182e4p-55},
    {0x1.33c08b26416ffp+0, 0x1.32721843659a6p-54},
    {0x1.371a7373aa9cbp+0, -0x1.63aeabf42eae2p-54},
    {0x1.3a7db34e59ff7p+0, -0x1.5e436d661f5e3p-56},
    {0x1.3dea64c123422p+0, 0x1.ada0911f09ebcp-55},
    {0x1.4160a21f72e2ap+0, -0x1.ef3691c309278p-58},
    {0x1.44e086061892dp+0, 0x1.89b7a04ef80d0p-59},
    {0x1.486a2b5c13cd0p+0, 0x1.3c1a3b69062f0p-56},
    {0x1.4bfdad5362a27p+0, 0x1.d4397afec42e2p-56},
    {0x1.4f9b2769d2ca7p+0, -0x1.4b309d25957e3p-54},
    {0x1.5342b569d4f82p+0, -0x1.07abe1db13cadp-55},
    {0x1.56f4736b527dap+0, 0x1.9bb2c011d93adp-54},
    {0x1.5ab07dd485429p+0, 0x1.6324c054647adp-54},
    {0x1.5e76f15ad2148p+0, 0x1.ba6f93080e65ep-54},
    {0x1.6247eb03a5585p+0, -0x1.383c17e40b497p-54},
    {0x1.6623882552225p+0, -0x1.bb60987591c34p-54},
    {0x1.6a09e667f3bcdp+0, -0x1.bdd3413b26456p-54},
    {0x1.6dfb23c651a2fp+0, -0x1.bbe3a683c88abp-57},
    {0x1.71f75e8ec5f74p+0, -0x1.16e4786887a99p-55},
    {0x1.75feb564267c9p+0, -0x1.0245957316dd3p-54},
    {0x1.7a11473eb0187p+0, -0x1.41577ee04992fp-55},
    {0x1.7e2f336cf4e62p+0, 0x1.05d02ba15797ep-56},
    {0x1.82589994cce13p+0, -0x1.d4c1dd41532d8p-54},
    {0x1.868d99b4492edp+0, -0x1.fc6f89bd4f6bap-54},
    {0x1.8ace5422aa0dbp+0, 0x1.6e9f156864b27p-54},
    {0x1.8f1ae99157736p+0, 0x1.5cc13a2e3976cp-55},
    {0x1.93737b0cdc5e5p+0, -0x1.75fc781b57ebcp-57},
    {0x1.97d829fde4e50p+0, -0x1.d185b7c1b85d1p-54},
    {0x1.9c49182a3f090p+0, 0x1.c7c46b071f2bep-56},
    {0x1.a0c667b5de565p+0, -0x1.359495d1cd533p-54},
    {0x1.a5503b23e255dp+0, -0x1.d2f6edb8d41e1p-54},
    {0x1.a9e6b5579fdbfp+0, 0x1.0fac90ef7fd31p-54},
    {0x1.ae89f995ad3adp+0, 0x1.7a1cd345dcc81p-54},
    {0x1.b33a2b84f15fbp+0, -0x1.2805e3084d708p-57},
    {0x1.b7f76f2fb5e47p+0, -0x1.5584f7e54ac3bp-56},
    {0x1.bcc1e904bc1d2p+0, 0x1.23dd07a2d9e84p-55},
    {0x1.c199bdd85529cp+0, 0x1.11065895048ddp-55},
    {0x1.c67f12e57d14bp+0, 0x1.2884dff483cadp-54},
    {0x1.cb720dcef9069p+0, 0x1.503cbd1e949dbp-56},
    {0x1.d072d4a07897cp+0, -0x1.cbc3743797a9cp-54},
    {0x1.d5818dcfba487p+0, 0x1.2ed02d75b3707p-55},
    {0x1.da9e603db3285p+0, 0x1.c2300696db532p-54},
    {0x1.dfc97337b9b5fp+0, -0x1.1a5cd4f184b5cp-54},
    {0x1.e502ee78b3ff6p+0, 0x1.39e8980a9cc8fp-55},
    {0x1.ea4afa2a490dap+0, -0x1.e9c23179c2893p-54},
    {0x1.efa1bee615a27p+0, 0x1.dc7f486a4b6b0p-54},
    {0x1.f50765b6e4540p+0, 0x1.9d3e12dd8a18bp-54},
    {0x1.fa7c1819e90d8p+0, 0x1.74853f3a5931ep-55},
};

// floor(2^(j/64) 2^176), 192-bit little-endian limbs, j = 0 .. 63.
__constant__ uint64_t EXP64_T_FX[64][3] = {
    {0x0ull, 0x0ull, 0x1000000000000ull},
    {0xbde93d70a2cabc5cull, 0xee6f7caca4f7a29ull, 0x102c9a3e77806ull},
    {0x17fe53e3495f7df4ull, 0x43ae7c548eb68ca4ull, 0x1059b0d315857ull},
    {0x2b041b2d6829d899ull, 0x808c35f25d9427faull, 0x10874518759bcull},
    {0x8364291408b3ceb0ull, 0xf6298b92b71842a9ull, 0x10b5586cf9890ull},
    {0x52ac4b358b1129e9ull, 0x2020742e4f8af6a5ull, 0x10e3ec32d3d1aull},
    {0xeac5cc47ab166ee5ull, 0xa4ebbf1aed9318cull, 0x111301d0125b5ull},
    {0x1844b389bea7aedull, 0xfb34101943b2586dull, 0x11429aaea92ddull},
    {0x792035509ff7d758ull, 0xadcdf7c8c50eb14aull, 0x1172b83c7d517ull},
    {0x5a6c30724d5cfae3ull, 0x53cb698f692d1c83ull, 0x11a35beb6fcb7ull},
    {0xa98b42206e46166cull, 0xa7805b8028990f07ull, 0x11d4873168b9aull},
    {0xfc487d21c2b8400ull, 0x63b8eeb02950929dull, 0x12063b88628cdull},
    {0x93b0328566902df6ull, 0x866c1fadb1c15cb5ull, 0x12387a6e75623ull},
    {0x9dce4e9186ddd5ffull, 0xd257a673281d3b24ull, 0x126b4565e27cdull},
    {0xbca890ac08d203feull, 0x12c25d15f5a24aa3ull, 0x129e9df51fdeeull},
    {0x4589c1cd1b3e4018ull, 0xb40091d536d07538ull, 0x12d285a6e4030ull},
    {0xedecbc27343629f5ull, 0x52de8d5a46305c85ull, 0x1306fe0a31b71ull},
    {0xf95d1593039539d9ull, 0xf4c9c8610d96696bull, 0x133c08b26416full},
    {0x7e3e12516bf9c699ull, 0xaa7145502f454798ull, 0x1371a7373aa9cull},
    {0x36163fe2f852ceebull, 0x6ea1bc9299e0a1d3ull, 0x13a7db34e59ffull},
    {0xfba2cb82b8244267ull, 0x235b41223e13d773ull, 0x13dea64c12342ull},
    {0xb352f0540e6ba056ull, 0x9f84325b8f3db61full, 0x14160a21f72e2ull},
    {0xbd4f3b48709b7859ull, 0xd03136f409df019full, 0x144e086061892ull},
    {0xc3dd75ce8757f780ull, 0x13c1a3b69062f03ull, 0x1486a2b5c13cdull},
    {0xe0363ba2e159c579ull, 0x71d4397afec42e20ull, 0x14bfdad5362a2ull},
    {0xe55e028497a329a7ull, 0x6ad33d8b69aa073eull, 0x14f9b2769d2caull},
    {0xf4e672a3e429805bull, 0x1df0a83c49d86a63ull, 0x15342b569d4f8ull},
    {0xf2f5ab3d801d7cull, 0xa66ecb004764eb3cull, 0x156f4736b527dull},
    {0x5d88d7c81280e069ull, 0x958c93015191eb34ull, 0x15ab07dd48542ull},
    {0xa06548a05829e853ull, 0x86e9be4c20399766ull, 0x15e76f15ad214ull},
    {0xbb1ceaf9f732275bull, 0x4b1f0fa06fd2da42ull, 0x16247eb03a558ull},
    {0xa337f4dc0a3adf17ull, 0x49127d9e29b8f314ull, 0x1662388255222ull},
    {0x7d3e3adec1751277ull, 0xc908b2fb1366ea95ull, 0x16a09e667f3bcull},
    {0x34b3f11577ceefbeull, 0xef220e2cbe1bbaa8ull, 0x16dfb23c651a2ull},
    {0xcb434b562d9e8a20ull, 0x3dd2370f2ef0acd6ull, 0x171f75e8ec5f7ull},
    {0x71805e61a17b954ull, 0x8bf6e9aa33a48b27ull, 0x175feb564267cull},
    {0x5ef42b6697796053ull, 0x6d7d51023f6cda1full, 0x17a11473eb018ull},
    {0x70a1427f8fcdf5f3ull, 0x2105d02ba15797e1ull, 0x17e2f336cf4e6ull},
    {0xf6ad65cbbac0f53ull, 0x28acf88afab34a01ull, 0x182589994cce1ull},
    {0x7484d73f136fb577ull, 0xc80e41d90ac25170ull, 0x1868d99b4492eull},
    {0x3e6ed61f2733304aull, 0xb5ba7c55a192c9bbull, 0x18ace5422aa0dull},
    {0x4efc9b4ae1458ae9ull, 0x62b982745c72ed80ull, 0x18f1ae9915773ull},
    {0xd2fc4af581b63e83ull, 0x4f4501c3f2540a22ull, 0x193737b0cdc5eull},
    {0xedb9d7144b6f6818ull, 0xf8b9e920f91e8bd7ull, 0x197d829fde4e4ull},
    {0x8ddade50c217186cull, 0x1c7c46b071f2be5ull, 0x19c49182a3f09ull},
    {0xaa0422a8da7d4512ull, 0x4b29ada8b8cab349ull, 0x1a0c667b5de56ull},
    {0x8050a405381703efull, 0xc8b424491caf87bcull, 0x1a5503b23e255ull},
    {0x58b571cf465caf07ull, 0xf43eb243bdff4c4cull, 0x1a9e6b5579fdbull},
    {0x7fbc3ae675ea440bull, 0xd5e8734d1773205aull, 0x1ae89f995ad3aull},
    {0x575781dbb49b1237ull, 0xaf6bfd0e7bd947c2ull, 0x1b33a2b84f15full},
    {0x54c8903c356e4b62ull, 0x6eaa7b081ab53c53ull, 0x1b7f76f2fb5e4ull},
    {0xd0b20287092bd59bull, 0x2247ba0f45b3d08cull, 0x1bcc1e904bc1dull},
    {0x679444964a366612ull, 0xc2220cb12a091ba6ull, 0x1c199bdd85529ull},
    {0x1dd9e6b151a6d1f9ull, 0xb4a2137fd20f2b30ull, 0x1c67f12e57d14ull},
    {0x61d9559ac0cb6dd3ull, 0x91503cbd1e949db7ull, 0x1cb720dcef906ull},
    {0x8fbbfc625f09f4ccull, 0xb8d0f22f21a158e1ull, 0x1d072d4a07897ull},
    {0xa9f589f559c0876full, 0x725da05aeb66e0dcull, 0x1d5818dcfba48ull},
    {0xf6246f0ec614ec95ull, 0x5708c01a5b6d4c97ull, 0x1da9e603db328ull},
    {0x7225a944efd5bb55ull, 0xeb968cac39ed291bull, 0x1dfc97337b9b5ull},
    {0xf49659e1693be17aull, 0x6273d130153991e8ull, 0x1e502ee78b3ffull},
    {0x1f86dea20610ceeeull, 0x9858f73a18f5db30ull, 0x1ea4afa2a490dull},
    {0x6dd5d229ff68e46full, 0x7771fd21a92dac1full, 0x1efa1bee615a2ull},
    {0xff99000dfc4352baull, 0x674f84b762862baull, 0x1f50765b6e454ull},
    {0xdc060c36f7650b4cull, 0x82e90a7e74b263c1ull, 0x1fa7c1819e90dull},
};

// floor(ln2/64 2^176).
__constant__ uint64_t EXP64_C_FX[3] = {0xcbdabd03cd0c99caull, 0x3de6af278ece600full, 0x2c5c85fdf47ull};

// 1/n!, binary64, n = 3 .. 11.
constexpr double INV_FACT[12] = {0, 0, 0,
                                 0x1.5555555555555p-3, 0x1.5555555555555p-5, 0x1.1111111111111p-7,
                                 0x1.6c16c16c16c17p-10, 0x1.a01a01a01a01ap-13, 0x1.a01a01a01a01ap-16,
                                 0x1.71de3a556c734p-19, 0x1.27e4fb7789f5cp-22, 0x1.ae64567f544e4p-26};

// ---- 192-bit unsigned fixed point (value = integer / 2^176) ----
struct U192 {
  uint64_t w[3];
};

__device__ __forceinline__ U192 u_add(U192 a, U192 b) {
  U192 r;
  unsigned __int128 t = (unsigned __int128)a.w[0] + b.w[0];
  r.w[0] = (uint64_t)t;
  t = (unsigned __int128)a.w[1] + b.w[1] + (uint64_t)(t >> 64);
  r.w[1] = (uint64_t)t;
  r.w[2] = a.w[2] + b.w[2] + (uint64_t)(t >> 64);
  return r;
}

__device__ __forceinline__ U192 u_sub(U192 a, U192 b) {  // a >= b
  U192 r;
  const uint64_t b0 = a.w[0] < b.w[0] ? 1 : 0;
  r.w[0] = a.w[0] - b.w[0];
  const uint64_t t1 = a.w[1] - b.w[1];
  const uint64_t b1 = (a.w[1] < b.w[1] || (a.w[1] == b.w[1] && b0)) ? 1 : 0;
  r.w[1] = t1 - b0;
  r.w[2] = a.w[2] - b.w[2] - b1;
  return r;
}

__device__ __forceinline__ bool u_less(U192 a, U192 b) {
  if (a.w[2] != b.w[2]) return a.w[2] < b.w[2];
  if (a.w[1] != b.w[1]) return a.w[1] < b.w[1];
  return a.w[0] < b.w[0];
}

// (a b) / 2^176, truncated (both below 2^16 in value).
__device__ __forceinline__ U192 u_mul(U192 a, U192 b) {
  uint64_t p[6] = {0, 0, 0, 0, 0, 0};
  for (int i = 0; i < 3; ++i) {
    uint64_t carry = 0;
    for (int j = 0; j < 3; ++j) {
      const unsigned __int128 t = (unsigned __int128)a.w[i] * b.w[j] + p[i + j] + carry;
      p[i + j] = (uint64_t)t;
      carry = (uint64_t)(t >> 64);
    }
    p[i + 3] = carry;
  }
  U192 r;
  for (int i = 0; i < 3; ++i) r.w[i] = (p[i + 2] >> 48) | (p[i + 3] << 16);
  return r;
}

// a m for a small integer m (the product stays below 2^192).
__device__ __forceinline__ U192 u_mul_small(U192 a, uint64_t m) {
  U192 r;
  uint64_t carry = 0;
  for (int i = 0; i < 3; ++i) {
    const unsigned __int128 t = (unsigned __int128)a.w[i] * m + carry;
    r.w[i] = (uint64_t)t;
    carry = (uint64_t)(t >> 64);
  }
  return r;
}

// a / n, truncated, for 1 <= n < 2^32 (long division in 32-bit digits).
__device__ __forceinline__ U192 u_div_small(U192 a, uint32_t n) {
  U192 r;
  uint64_t rem = 0;
  for (int i = 2; i >= 0; --i) {
    const uint64_t hi = (rem << 32) | (a.w[i] >> 32);
    const uint64_t qh = hi / n;
    rem = hi - qh * n;
    const uint64_t lo = (rem << 32) | (a.w[i] & 0xffffffffull);
    const uint64_t ql = lo / n;
    rem = lo - ql * n;
    r.w[i] = (qh << 32) | ql;
  }
  return r;
}

// a.w[i] for 0 <= i < 3 (0 otherwise), by selection rather than an indexed access, so
// nothing of a U192 lives in scratch memory.
__device__ __forceinline__ uint64_t u_word(const U192 &a, int i) {
  return i == 0 ? a.w[0] : i == 1 ? a.w[1] : i == 2 ? a.w[2] : 0ull;
}

__device__ __forceinline__ bool u_bit(const U192 &a, int pos) {
  return (u_word(a, pos >> 6) >> (pos & 63)) & 1ull;
}

__device__ __forceinline__ bool u_any_below(const U192 &a, int pos) {  // a bit below position pos
  for (int i = 0; i < 3; ++i) {
    const int lo = 64 * i;
    if (pos <= lo) break;
    const uint64_t mask = pos >= lo + 64 ? ~0ull : ((1ull << (pos - lo)) - 1ull);
    if (a.w[i] & mask) return true;
  }
  return false;
}

__device__ __forceinline__ uint64_t u_shr_low(const U192 &a, int s) {  // low 64 bits of a >> s
  const int i = s >> 6, b = s & 63;
  uint64_t v = u_word(a, i) >> b;
  if (b) v |= u_word(a, i + 1) << (64 - b);
  return v;
}

__device__ __forceinline__ int u_top_bit(const U192 &a) {
  for (int i = 2; i >= 0; --i)
    if (a.w[i]) return 64 * i + 63 - __builtin_clzll(a.w[i]);
  return -1;
}

// Second stage: e^x to about 2^-165, rounded to binary64 (N, j, k as in the first stage).
__device__ __noinline__ double exp64_fixed(double x, int N, int j, int k) {
  // |x| = m 2^e exactly; X = |x| 2^176 (truncated below 2^-176 for tiny |x|)
  int ex;
  const double f = __builtin_frexp(__builtin_fabs(x), &ex);  // f in [0.5, 1)
  const uint64_t m = (uint64_t)__builtin_ldexp(f, 53);
  const int s = ex - 53 + 176;
  U192 X = {{0, 0, 0}};
  if (s >= 0) {  // s < 192 - 53: the two words below stay inside X
    const int i = s >> 6, b = s & 63;
    const uint64_t lo = m << b, hi = b ? m >> (64 - b) : 0ull;
    X.w[0] = i == 0 ? lo : 0ull;
    X.w[1] = i == 1 ? lo : i == 0 ? hi : 0ull;
    X.w[2] = i == 2 ? lo : i == 1 ? hi : 0ull;
  } else if (s > -64) {
    X.w[0] = m >> (-s);
  }
  const U192 C = {{EXP64_C_FX[0], EXP64_C_FX[1], EXP64_C_FX[2]}};
  const U192 NC = u_mul_small(C, (uint64_t)(N < 0 ? -N : N));
  // r = x - N ln2/64; x and N share their sign
  bool neg = x < 0;
  U192 R;
  if (u_less(X, NC)) {
    R = u_sub(NC, X);
    neg = !neg;
  } else {
    R = u_sub(X, NC);
  }
  // e^r = sum_n r^n / n!, the sign of r^n alternating when r < 0
  U192 S = {{0, 0, (uint64_t)1 << 48}};  // 1
  U192 T = S;
  for (int n = 1; n <= 20; ++n) {
    T = u_div_small(u_mul(T, R), (uint32_t)n);
    S = (neg && (n & 1)) ? u_sub(S, T) : u_add(S, T);
  }
  const U192 Tj = {{EXP64_T_FX[j][0], EXP64_T_FX[j][1], EXP64_T_FX[j][2]}};
  const U192 Y = u_mul(Tj, S);  // e^x / 2^k, in [0.99, 2)
  if (k >= -1021) {
    const int L = u_top_bit(Y);  // 175 or 176
    uint64_t sig = u_shr_low(Y, L - 52);
    const bool guard = u_bit(Y, L - 53), sticky = u_any_below(Y, L - 53);
    sig += (guard && (sticky || (sig & 1ull))) ? 1ull : 0ull;
    return __builtin_ldexp((double)sig, L - 52 - 176 + k);
  }
  const int sh = 176 - (k + 1074);  // the quantum 2^-1074 in units of 2^-176 2^-k
  uint64_t n = u_shr_low(Y, sh);
  const bool guard = u_bit(Y, sh - 1), sticky = u_any_below(Y, sh - 1);
  n += (guard && (sticky || (n & 1ull))) ? 1ull : 0ull;
  return __builtin_ldexp((double)n, -1074);
}

// First stage for |x| < 2^-27 (the low components of an expansion): e^x = (1 + x) +
// x^2/2 + x^3/6 + O(2^-110), 1 + x split exactly into a double-double; the same margin
// test as the general first stage.  Returns true and sets y when it decides the rounding.
__device__ __forceinline__ bool exp64_first_small(double x, double &y) {
  const DD a = dd_sum(1.0, x);
  const double t = a.lo + (x * x) * (0.5 + x * INV_FACT[3]);
  const double lo = a.hi + (t - 0x1p-69), hi = a.hi + (t + 0x1p-69);
  y = x == 0.0 ? 1.0 : lo;
  return x == 0.0 || lo == hi;
}

// First stage of the correctly rounded binary64 e^x, any x: returns true and sets y when
// the double-double value decides the rounding (NaN, overflow and underflow included).
// Special arguments are replaced by 0 for the arithmetic and their results selected at
// the end; results below 2^-1021 take a branch that is uniform across the wavefront, so
// the common path runs without one.
__device__ __forceinline__ bool exp64_first(double x, const double (*__restrict__ tdd)[2], double &y) {
  const bool nan = x != x, over = x > 710.0, under = x < -746.0;
  const bool special = nan || over || under;
  const double xs = special ? 0.0 : x;
  const double Nd = __builtin_rint(xs * EXP64_INV);
  const int N = (int)Nd;
  const int j = N & 63;
  const int k = (N - j) / 64;
  // r = x - N ln2/64 as a double-double: N L1 is exact and so is x - N L1
  const double t = xs - Nd * EXP64_L1;
  const double p2 = Nd * EXP64_L2;
  const double e2 = __builtin_fma(Nd, EXP64_L2, -p2);
  DD r = dd_sum(t, -p2);
  r = dd_fast_sum(r.hi, (r.lo - e2) - Nd * EXP64_L3);
  const double rh = r.hi, rl = r.lo;
  // e^r = 1 + r + r^2/2 + r^3 q(r), q = 1/3! + r/4! + ... + r^6/9! in binary64
  double q = INV_FACT[9];
  for (int n = 8; n >= 3; --n) q = __builtin_fma(q, rh, INV_FACT[n]);
  const double r2h = rh * rh;
  const double r2l = __builtin_fma(rh, rh, -r2h) + 2.0 * rh * rl;
  const double low = rl + 0.5 * r2l + q * (r2h * rh);
  // P = 1 + (r + r^2/2) + low: r + r^2/2 split exactly, 1 + its high part exactly
  const DD s2 = dd_sum(rh, 0.5 * r2h);
  const DD o = dd_fast_sum(1.0, s2.hi);
  const double pl = o.lo + (s2.lo + low);
  // Y = 2^(j/64) P, left unnormalized (|Y.lo| < 2^-24 |Y.hi|): the margin test below
  // takes it as it is; the rounding to a multiple of 2^-1074 normalizes it first
  const double th = tdd[j][0], tl = tdd[j][1];
  const double p = th * o.hi;
  const DD Y = {p, __builtin_fma(th, o.hi, -p) + (th * pl + tl * o.hi)};
  const double e = 0x1p-69 * Y.hi;
  const double lo = Y.hi + (Y.lo - e), hi = Y.hi + (Y.lo + e);
  double v = __builtin_ldexp(lo, k);
  bool ok = lo == hi;
  const bool sub = k < -1021;
  if (__builtin_expect(__any(sub), 0)) {
    if (sub) {  // results below 2^-1021: round to a multiple of 2^-1074
      const DD Z = dd_fast_sum(Y.hi, Y.lo);
      const double zh = __builtin_ldexp(Z.hi, k + 1074), zl = __builtin_ldexp(Z.lo, k + 1074);
      const double i = __builtin_rint(zh);
      const double d = (zh - i) + zl;
      const double ez = 0x1p-69 * zh;
      ok = true;
      double w = 0.0;
      if (d < 0.5 - ez && d > -0.5 + ez) w = i;
      else if (d > 0.5 + ez) w = i + 1.0;
      else if (d < -0.5 - ez) w = i - 1.0;
      else ok = false;
      v = __builtin_ldexp(w, -1074);
    }
  }
  const double sv = nan ? x + x : (over ? __builtin_inf() : 0.0);
  y = special ? sv : v;
  return special || ok;
}

// Second stage for the arguments the first leaves undecided (about one in 2^16).
__device__ __noinline__ double exp64_second(double x) {
  const int N = (int)__builtin_rint(x * EXP64_INV);
  const int j = N & 63;
  return exp64_fixed(x, N, j, (N - j) / 64);
}

// Exp-MCN of one element: h = (e^x_0), then h = ScalingN(h, e^x_i) with expand.
template <int N, int M>
__device__ __forceinline__ void exp64_chain(const double (&h)[M], const double (&ex)[N], double (&out)[N]) {
  if constexpr (M == N) {
#pragma unroll
    for (int c = 0; c < N; ++c) out[c] = h[c];
  } else {
    double g[M + 1];
    scaling_n<double, M, M + 1>(h, ex[M], g);
    exp64_chain<N, M + 1>(g, ex, out);
  }
}

constexpr int EXP64_THREADS = 256;

template <int NC>
__global__ __launch_bounds__(EXP64_THREADS) void exp64_kernel(const double *__restrict__ x,
                                                              double *__restrict__ out, int64_t n) {
  __shared__ double tdd[64][2];
  if (threadIdx.x < 128) tdd[threadIdx.x >> 1][threadIdx.x & 1] = EXP64_T_DD[threadIdx.x >> 1][threadIdx.x & 1];
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * EXP64_THREADS;
  int64_t i = (int64_t)blockIdx.x * EXP64_THREADS + threadIdx.x;
  if (i >= n) return;
  double cur[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) cur[c] = x[c * n + i];
  while (true) {
    // the next element's loads go out before this one's arithmetic (the last lane
    // iteration re-reads its own element)
    const int64_t nx = i + stride;
    const bool more = nx < n;
    const int64_t ni = more ? nx : i;
    double nxt[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) nxt[c] = x[c * n + ni];
    // the short first stage when every lane's argument is small (the general one is
    // valid for small arguments too), then the second stage where a lane needs it
    double ex[NC];
    bool okc[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      if (__all(__builtin_fabs(cur[c]) < 0x1p-27))
        okc[c] = exp64_first_small(cur[c], ex[c]);
      else
        okc[c] = exp64_first(cur[c], tdd, ex[c]);
    }
    bool ok = true;
#pragma unroll
    for (int c = 0; c < NC; ++c) ok = ok && okc[c];
    if (__builtin_expect(__any(!ok), 0)) {
#pragma unroll
      for (int c = 0; c < NC; ++c)
        if (!okc[c]) ex[c] = exp64_second(cur[c]);
    }
    const double h0[1] = {ex[0]};
    double r[NC];
    exp64_chain<NC, 1>(h0, ex, r);
#pragma unroll
    for (int c = 0; c < NC; ++c) out[c * n + i] = r[c];
    if (!more) break;
    i = nx;
#pragma unroll
    for (int c = 0; c < NC; ++c) cur[c] = nxt[c];
  }
}

template <int NC>
hipError_t exp64_launch(int64_t n, const void *x, void *out, hipStream_t s) {
  int64_t blocks = (n + EXP64_THREADS - 1) / EXP64_THREADS;
  if (blocks > 16384) blocks = 16384;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL((exp64_kernel<NC>), dim3((unsigned)blocks), dim3(EXP64_THREADS), 0, s, (const double *)x,
                     (double *)out, n);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_exp_f64(int nc, int64_t n, const void *x, void *out, hipStream_t stream) {
  switch (nc) {
    case 1: return exp64_launch<1>(n, x, out, stream);
    case 2: return exp64_launch<2>(n, x, out, stream);
    case 3: return exp64_launch<3>(n, x, out, stream);
    case 4: return exp64_launch<4>(n, x, out, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace mcf
