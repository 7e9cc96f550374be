// Test-only cross-check: evaluates rocRAND's independent Philox4x32-10
// bijection (ten_rounds of rocrand_philox4x32_10.h) on (counter, key) pairs read
// from stdin as little-endian uint32 sextuples, writing the 4 output words of
// each pair to stdout.  Built with the host compiler; never linked into the
// library or the oracle.
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdint>
#include <cstdio>

struct Engine : rocrand_device::philox4x32_10_engine {
    uint4 bijection(uint4 c, uint2 k) { return ten_rounds(c, k); }
};

int main()
{
    Engine e;
    uint32_t in[6];
    while (std::fread(in, sizeof(uint32_t), 6, stdin) == 6) {
        uint4 c = {in[0], in[1], in[2], in[3]};
        uint2 k = {in[4], in[5]};
        uint4 r = e.bijection(c, k);
        uint32_t out[4] = {r.x, r.y, r.z, r.w};
        std::fwrite(out, sizeof(uint32_t), 4, stdout);
    }
    return 0;
}
