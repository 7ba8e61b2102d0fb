"""MI355X-native relational GNN layers (RGCN, RGAT, HGT) behind the C ABI of
librgnn.so.  `paper_2301_06284_amd.rgnn` is the ctypes binding; it loads the
built HIP library and fails loudly when it is missing."""
