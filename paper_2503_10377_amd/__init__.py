"""libsppo: sequence-chunked causal attention (forward + backward) with
per-chunk activation offload, for MI355X (gfx950).

``sppo``           ctypes binding of the C ABI in include/sppo.h
``chunked``        the chunk loop (forward walk with offload, reverse backward
                   walk with prefetch) over that ABI
``chunked_layer``  the same walk for a whole pre-LayerNorm transformer layer
``ring``           the device staging arena for offloaded chunks and its planner
``pacing``         keeps the host a bounded number of chunks ahead of the device
``inputs``         seeded synthetic inputs
``build``          in-tree hipcc build of libsppo.so
"""
