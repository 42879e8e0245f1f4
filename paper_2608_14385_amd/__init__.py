"""MI355X-native DeaMoE decode layer: HIP kernels behind a C ABI (libdeamoe.so).

`paper_2608_14385_amd.deamoe` is the Python binding of the C ABI;
`paper_2608_14385_amd.workloads` draws seeded synthetic inputs.
"""
