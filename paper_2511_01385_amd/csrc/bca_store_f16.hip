// bca_store_f16.hip -- the fused layer kernels of bca_kernels.hpp for StoreF16 rows.
#include "bca_kernels.hpp"

namespace rdfft {

BcaStoreTables bca_tables_f16() { return make_store_tables<StoreF16>(); }

}  // namespace rdfft
