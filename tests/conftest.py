def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: runs the HIP library on an MI355X")
