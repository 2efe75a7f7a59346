"""CPU oracle (test infrastructure only): plain double-precision C of one
GraphSAGE layer's forward and backward feature propagation, used to check
the GPU library.  The GPU library never imports or links it."""
