// Host entry points over the integer maps the contraction kernels use to
// distribute tiles and stream-K iterations (pk_partition.hpp), built by the
// CPU tests with hipcc for the host only: the tests check the very functions
// the kernels call, not a copy of their formulas.
#include "../paper_1904_05347_amd/csrc/pk_partition.hpp"

extern "C" {

int shim_sk_start(int T, int G, int nkb, int g) { return pk::StreamK{T, G, nkb}.start(g); }
int shim_sk_owner(int T, int G, int nkb, int i) { return pk::StreamK{T, G, nkb}.owner(i); }
int shim_sk_slot(int T, int G, int nkb, int g, int t) { return pk::StreamK{T, G, nkb}.slot(g, t); }
int shim_sk_logical(int b, int G, int xcds) { return pk::sk_logical(b, G, xcds); }
int shim_xcd_tile(int pid, int num, int xcds) { return pk::xcd_tile(pid, num, xcds); }
void shim_tile_of(int tiles_m, int tiles_n, int group_m, int t, int *tm, int *tn)
{
    pk::tile_of_ints(tiles_m, tiles_n, group_m, t, *tm, *tn);
}

}  // extern "C"
