// pk_registry.hip -- the list of every compiled configuration.
#include <vector>

#include "pk_configs.hpp"

namespace pk {

const Config *configs_gemm_nn(int *count);
const Config *configs_gemm_tn(int *count);
const Config *configs_gemm_nt(int *count);
const Config *configs_gemm_tt(int *count);
const Config *configs_conv(int *count);
const Config *configs_direct(int *count);
const Config *configs_direct_tiled(int *count);

const Config *configs(int *count)
{
    static const std::vector<Config> all = [] {
        std::vector<Config> v;
        for (auto group : {configs_gemm_nn, configs_gemm_tn, configs_gemm_nt, configs_gemm_tt, configs_conv, configs_direct,
                           configs_direct_tiled}) {
            int n = 0;
            const Config *c = group(&n);
            v.insert(v.end(), c, c + n);
        }
        return v;
    }();
    *count = (int)all.size();
    return all.data();
}

}  // namespace pk
