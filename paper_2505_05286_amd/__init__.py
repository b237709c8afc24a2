"""MI355X-native serving instance for agentic Text-to-SQL workflows.

``hxf`` is the ctypes binding of ``libhxf.so`` (C ABI in ``include/``);
``device`` places a model's weights, KV pool and workspace in HBM with
PyTorch and binds them to an instance.
"""
